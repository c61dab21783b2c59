/*
 * nova.h -- C ABI of libnova: the single-GPU hot path of agentic VLM serving on MI355X (gfx950).
 *
 * A request is a screenshot plus an instruction (the paper's Sec. 2.1).  It passes through three
 * stages: vision encode (ViT + adapter), LLM prefill over [visual embeddings ; instruction
 * tokens] which builds the KV cache, and LLM decode, one greedy token per batched step
 * (Sec. 2.1, Sec. 2.2; in-flight decode batching, Sec. 3.4).  The stages run concurrently on
 * disjoint compute-unit partitions chosen before each forward pass (Sec. 3.2.2, Sec. 3.4), and
 * vision-encoder layers can be streamed from pinned host memory into K device slots (Sec. 3.5,
 * Eq. 7).
 *
 * Conventions for every call:
 *  - Return value: NOVA_OK (0) or a negative status; nova_last_error() then describes the failure
 *    (thread-local string).  Nothing is thrown across the ABI.
 *  - Pointers named "device" must point to GPU memory of the current device, 256-byte aligned.
 *    The caller owns all device and pinned-host memory (weights, KV pools, workspaces,
 *    inputs, outputs); the library never frees caller memory and never allocates device
 *    memory in the stage calls.  The library owns only its streams and events.
 *  - Stage calls are asynchronous on the given stream (0 = the null stream): errors in argument
 *    checks and kernel launches are reported at once; faults inside kernels surface at the
 *    caller's next synchronisation.
 *  - Element types: weights are bf16 (uint16 bit patterns).  Activations (stage inputs/outputs,
 *    KV cache) are bf16 when the model's act == NOVA_ACT_BF16 and fp32 when NOVA_ACT_F32.
 *    Logits are always fp32, token ids and block tables int32.
 *  - Threading: one thread per stage may call concurrently (vision, prefill, decode workers,
 *    Sec. 3.1).  A model object may be shared by the prefill and decode threads (they share
 *    weights, Sec. 3.1); nova_vit_encode with offload and nova_prefetch_layer on one nova_vit
 *    must come from one thread.
 */
#ifndef NOVA_H
#define NOVA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* nova_stream_t; /* a hipStream_t */

enum {
  NOVA_OK = 0,
  NOVA_EINVAL = -1,       /* invalid argument (shape, pointer, alignment, range) */
  NOVA_ENOKV = -2,        /* block table does not cover the requested positions */
  NOVA_EHIP = -3,         /* a HIP runtime call or kernel launch failed */
  NOVA_EUNSUPPORTED = -4, /* configuration outside what the kernels implement */
  NOVA_ENOSPACE = -5      /* workspace smaller than nova_*_workspace_bytes() */
};
enum { NOVA_STAGE_ENCODE = 0, NOVA_STAGE_PREFILL = 1, NOVA_STAGE_DECODE = 2 };
enum { NOVA_ACT_BF16 = 0, NOVA_ACT_F32 = 1 };
enum { NOVA_KIND_GEMM = 0, NOVA_KIND_ATTN = 1, NOVA_KIND_GEMV = 2, NOVA_KIND_DECODE_ATTN = 3, NOVA_KIND_MISC = 4 };

/* Last error message of this thread ("" if none). */
const char* nova_last_error(void);
/* Select the device and create the library's streams/events; call once per process. */
int nova_init(int device);
/* Destroy the library's streams and events (partition streams included). */
void nova_shutdown(void);
/* Number of compute units of the initialised device (256 on MI355X). */
int nova_device_cus(void);

/* ------------------------------------------------------------------ vision encoder (Sec. 2.1)
 * Pre-LN ViT: x0 = patches W_p^T + b_p + E_pos; each layer h = x + Attn(LN1 x) W_o^T + b_o,
 * y = h + GELU(LN2 h W_1^T + b_1) W_2^T + b_2 with bidirectional attention over all patches;
 * adapter: LN per patch, concatenation of each merge x merge patch group, Linear to out_hidden.
 */
typedef struct {
  int hidden, heads, mlp, layers;
  int patch, merge, out_hidden;   /* merge 1 (LN + Linear) or 2 (2x2 patch merge) */
  int image_h, image_w;           /* multiples of patch (and of patch*merge) */
  float eps;                      /* LayerNorm epsilon */
  int act;                        /* NOVA_ACT_BF16 or NOVA_ACT_F32 */
} nova_vit_config;

/* Packed weight blobs.  Every tensor is bf16, row-major, at the returned byte offset (256-byte
 * aligned) of its blob.  Linear weights are [out, in]; "in" is zero-padded to kpad / ip where noted.
 *  embed blob: 0 patch.w [hidden, kpad] (kpad = 3*patch^2 rounded up to 64, zero tail),
 *              1 patch.b [hidden], 2 pos [n_patches, hidden]
 *  layer blob: 0 ln1.g, 1 ln1.b [hidden], 2 qkv.w [3*hidden, hidden] (q | k | v, head-major),
 *              3 qkv.b [3*hidden], 4 o.w [hidden, hidden], 5 o.b, 6 ln2.g, 7 ln2.b,
 *              8 fc1.w [ip, hidden], 9 fc1.b [ip], 10 fc2.w [hidden, ip], 11 fc2.b
 *              (ip = mlp rounded up to 256; padded rows/columns are zero)
 *  head blob:  0 merge.ln.g, 1 merge.ln.b [hidden], 2 merge.w [out_hidden, merge^2*hidden], 3 merge.b
 * offsets must have room for 3 / 12 / 4 entries; *bytes receives the blob size. */
int nova_vit_embed_layout(const nova_vit_config* cfg, size_t* offsets, size_t* bytes);
int nova_vit_layer_layout(const nova_vit_config* cfg, size_t* offsets, size_t* bytes);
int nova_vit_head_layout(const nova_vit_config* cfg, size_t* offsets, size_t* bytes);

typedef struct {
  nova_vit_config cfg;
  const void* embed;        /* device embed blob */
  const void* head;         /* device head blob */
  const void* layers;       /* device: cfg.layers layer blobs back to back (resident), or NULL */
  /* Layer offload (Sec. 3.5): all layer blobs in pinned host memory, n_slots device slots. */
  const void* host_layers;  /* pinned host (hipHostMalloc): cfg.layers blobs back to back, or NULL */
  void* slots;              /* device: n_slots layer blobs back to back */
  int n_slots;              /* K, 2 <= K < layers */
} nova_vit_desc;

typedef struct nova_vit nova_vit;
/* Validate a descriptor and build a model handle (no device memory is allocated; with
 * offload, one copy stream and 2K events are created). */
int nova_vit_create(const nova_vit_desc* desc, nova_vit** out);
void nova_vit_destroy(nova_vit* vit);
/* Bytes of device workspace nova_vit_encode needs for this batch size. */
size_t nova_vit_workspace_bytes(const nova_vit* vit, int batch);

/* Vision encode of `batch` images.
 *  pixels: device bf16 [batch, image_h, image_w, 3] (HWC, values fed as is)
 *  out:    device act-type [batch, n_patches / merge^2, out_hidden]
 * With offload, every layer waits for its slot's copy and, once done, its slot receives layer
 * (l + K) mod L (Eq. 7), so the next call's first K layers are loaded during this one.  When K
 * does not divide L the layer-to-slot map rotates from one call to the next. */
int nova_vit_encode(nova_vit* vit, const void* pixels, int batch, void* out, void* ws, size_t ws_bytes,
                    nova_stream_t stream);

/* Swap logical ViT layer `layer` into a physical slot from pinned host memory on copy_stream
 * (0: the model's own copy stream), after the last compute use of that slot has finished
 * (Sec. 3.5: one event per physical layer guards both the copy and the compute).  No-op if the
 * layer is already in a slot.  The slot is the one holding layer (layer - K) mod L (the Eq. 7
 * ring), else an empty one, else slot layer mod K.  nova_vit_encode queues layers 0..K-1 this
 * way itself; calling it earlier moves those copies ahead of the first encode.  Returns
 * NOVA_EINVAL without offload. */
int nova_prefetch_layer(nova_vit* vit, int layer, nova_stream_t copy_stream);

/* Offload ring state, host side: slot_layer (may be NULL) receives the n_slots logical layers
 * the physical slots hold or are receiving (-1: none yet), copies (may be NULL) the number of
 * host-to-device layer copies issued since creation.  Over repeated encodes the ring issues L
 * copies per call (Eq. 7).  Returns NOVA_EINVAL without offload. */
int nova_vit_offload_state(const nova_vit* vit, int* slot_layer, unsigned long long* copies);

/* ------------------------------------------------------------------ LLM (Sec. 2.1, Sec. 3.4)
 * Decoder layer: RMSNorm -> q, k, v (no bias) -> rotary embedding (half-split pairs) -> causal
 * grouped-query attention -> W_o + residual -> RMSNorm -> SwiGLU MLP + residual; final RMSNorm,
 * untied LM head, greedy argmax (ties to the lowest id).
 */
typedef struct {
  int hidden, n_q, n_kv, head_dim, inter, vocab, layers;
  int block;         /* tokens per KV block; must be 16 */
  float rope_theta;
  float eps;         /* RMSNorm epsilon */
  int act;
} nova_llm_config;

/* layer blob: 0 rms1.g [hidden], 1 qkv.w [(n_q+2n_kv)*head_dim, hidden] (q | k | v, head-major),
 *             2 o.w [hidden, n_q*head_dim], 3 rms2.g [hidden],
 *             4 gu.w [2*ip, hidden]: gate and up rows interleaved in blocks of 8
 *               (rows 16j..16j+7 = gate rows 8j..8j+7, rows 16j+8..16j+15 = up rows 8j..8j+7),
 *             5 down.w [hidden, ip]      (ip = inter rounded up to 256; padding is zero)
 * head blob:  0 norm.g [hidden], 1 lm_head.w [vocab, hidden]
 * The embedding table is a separate device bf16 [vocab, hidden] array. */
int nova_llm_layer_layout(const nova_llm_config* cfg, size_t* offsets, size_t* bytes);
int nova_llm_head_layout(const nova_llm_config* cfg, size_t* offsets, size_t* bytes);

typedef struct {
  nova_llm_config cfg;
  const void* embed;    /* device bf16 [vocab, hidden] */
  const void* layers;   /* device: cfg.layers layer blobs back to back */
  const void* head;     /* device head blob */
} nova_llm_desc;
typedef struct nova_llm nova_llm;
int nova_llm_create(const nova_llm_desc* desc, nova_llm** out);
void nova_llm_destroy(nova_llm* llm);

/* Paged KV cache (PagedAttention-style blocks of 16 tokens), caller-owned device memory:
 *  k: [layers][num_blocks][n_kv][16][head_dim]   (rotated keys)
 *  v: [layers][num_blocks][n_kv][head_dim][16]   (values, transposed within each block)
 * Element type follows the model's act.  nova_kv_bytes() gives the size of each of k and v. */
typedef struct {
  void* k;
  void* v;
  int num_blocks;
} nova_kv;
size_t nova_kv_bytes(const nova_llm* llm, int num_blocks);

/* Device workspace for prefill of up to `seq` tokens, or decode of `batch` sequences whose
 * context never exceeds max_ctx tokens. */
size_t nova_llm_prefill_workspace_bytes(const nova_llm* llm, int seq);
size_t nova_llm_decode_workspace_bytes(const nova_llm* llm, int batch, int max_ctx);

/* Prefill one request (no batching of prefill, Sec. 3.4).
 *  vis:   device act-type [n_vis, hidden] visual embeddings (may be NULL when n_vis == 0)
 *  ids:   device int32 [n_text] instruction tokens, appended after the visual embeddings
 *  block_table: device int32 [ceil((n_vis+n_text)/16)] physical block of each 16 positions
 *  Writes the rotated K and V of positions 0..S-1 into kv, the greedy next token into
 *  next_id (device int32 [1]) and, if logits != NULL, the last-row logits (device fp32 [vocab]). */
int nova_llm_prefill(const nova_llm* llm, const void* vis, int n_vis, const int32_t* ids, int n_text,
                     const int32_t* block_table, const nova_kv* kv, int32_t* next_id, float* logits, void* ws,
                     size_t ws_bytes, nova_stream_t stream);

/* One in-flight-batched decode step for `batch` sequences (batch <= 32).
 *  ids, pos:     device int32 [batch]: token fed and its position (context becomes pos + 1)
 *  block_tables: device int32 [batch, max_blocks] (row b covers positions 0..pos[b])
 *  max_ctx:      an upper bound of pos[b] + 1 over the batch (sizes the attention split); a
 *                position outside 0..max_ctx - 1 is clamped into it (garbage out, no access
 *                outside the sequence's block-table row)
 *  Appends each sequence's K/V at pos[b], writes next_ids (device int32 [batch]) and, if
 *  logits != NULL, device fp32 [batch, vocab]. */
int nova_llm_decode(const nova_llm* llm, const int32_t* ids, const int32_t* pos, const int32_t* block_tables,
                    int max_blocks, int batch, int max_ctx, const nova_kv* kv, int32_t* next_ids, float* logits,
                    void* ws, size_t ws_bytes, nova_stream_t stream);

/* Allocation-free decode step, for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the same step as
 * nova_llm_decode, same arguments and results, with its workspace (activations, split-K partial
 * sums, arrival counters, attention split partials) taken from a library-owned static device
 * array of NOVA_DECODE_SCRATCH_BYTES bytes, which each GPU the library runs on holds until the
 * process ends.  Calls no hipMalloc, hipFree or other allocating routine.  The step clears what
 * must start at zero (argmax keys, arrival counters) in its own first kernel; the array keeps the
 * last call's contents otherwise.  Every call on one GPU uses that GPU's single array: calls that
 * overlap in time on one GPU (two streams, two threads) race on it and give wrong results, so
 * the caller serialises them.  A step whose workspace (nova_llm_decode_workspace_bytes) exceeds
 * NOVA_DECODE_SCRATCH_BYTES returns NOVA_ENOSPACE and launches nothing; the 28-layer 3584-wide
 * decoder at batch 32 needs about 9 MB. */
#define NOVA_DECODE_SCRATCH_BYTES (32u << 20)
int nova_llm_decode_noalloc(const nova_llm* llm, const int32_t* ids, const int32_t* pos, const int32_t* block_tables,
                            int max_blocks, int batch, int max_ctx, const nova_kv* kv, int32_t* next_ids,
                            float* logits, nova_stream_t stream);

/* ------------------------------------------------------------------ linear co-run study
 * The two-linear experiment behind the paper's choice of inter-CU partitioning (Sec. 3.2.1, its
 * linear co-run table, and Sec. 3.2.3): one linear layer out[M, N] += x[M, K] w[N, K]^T
 * (x, w device bf16 row-major, out device fp32, all 256-byte aligned), enqueued on `stream`,
 * with one of the kernels the stage calls use or the low-footprint pair of the intra-CU variant:
 *  NOVA_LINEAR_TILED       the encode / prefill GEMM (256x256 or 128x128 tiles as for the stages;
 *                          K % 64 == 0, N % 128 == 0)
 *  NOVA_LINEAR_TILED_SMALL the same GEMM held to 128x128 tiles of 4 waves (64 KB of LDS), so a
 *                          CU keeps room for another kernel's workgroups
 *  NOVA_LINEAR_THIN        the decode thin GEMM on the matrix cores (M <= 32, K % 256 == 0,
 *                          N % 64 == 0, and N large enough that K is not split on the stream's CUs)
 *  NOVA_LINEAR_THIN_VALU   the decode linear on the vector ALUs without LDS (M <= 4, K % 512 == 0)
 * Returns NOVA_EUNSUPPORTED outside those shapes. */
enum { NOVA_LINEAR_TILED = 0, NOVA_LINEAR_TILED_SMALL = 1, NOVA_LINEAR_THIN = 2, NOVA_LINEAR_THIN_VALU = 3 };
int nova_linear(int variant, const void* x, int M, int K, const void* w, int N, float* out, nova_stream_t stream);

/* ------------------------------------------------------------------ CU partitions (Sec. 3.2.2)
 * gfx950 deals a kernel's workgroups round-robin over its 8 XCDs, and a CU-mask bit i selects
 * CU slot i/32 of shader engine (i/8)%4 of XCD i%8.  A partition therefore never confines a
 * stage to whole XCDs (the other XCDs' share of its workgroups could not run); it takes the
 * same CU slots on every XCD.  32 CUs = one mask word = 4 CUs on each XCD, one per engine. */

/* XCD-balanced mask of n_cus CUs (a positive multiple of 8, <= 256) starting at CU slot
 * first_slot (0..31, per shader engine): mask bits for slots first_slot .. first_slot +
 * n_cus/8 - 1 on every XCD, engines interleaved.  mask must have room for 8 words. */
int nova_make_cu_mask(int n_cus, int first_slot, uint32_t* mask);

/* Give `stage` the CUs in cu_mask (mask_words 32-bit words, bit i = CU i as above) and return
 * in *out_stream a library-owned stream restricted to them (created with
 * hipExtStreamCreateWithCUMask on first use of that mask, default priority, then cached).
 * A new mask's complement (when it keeps a CU on every XCD) gets its stream created right
 * after it, so that a stage pair on complementary masks sits on different hardware dispatch
 * pipes and runs concurrently; pairs of other masks carry no such guarantee.  Stages given the
 * same partial mask share its stream; the whole-GPU mask has a separate stream per stage
 * (the three are created together).
 * Work enqueued afterwards on *out_stream starts only after everything previously enqueued on
 * the stage's prior partition stream (ordering across the switch, Sec. 3.4: partitions change
 * only between forward passes).  Host-synchronous; does not wait for the device.
 * An empty mask, a mask with no CU on some XCD, or stage out of range gives NOVA_EINVAL. */
int nova_set_stage_partition(int stage, const uint32_t* cu_mask, int mask_words, nova_stream_t* out_stream);

/* Diagnostic: launch n_workgroups single-wave workgroups on `stream`; workgroup i writes
 * (xcd << 16) | (shader_engine << 8) | cu of the compute unit it ran on into out[i]
 * (device uint32 [n_workgroups]).  Used to check that a partition stream stays on its CUs. */
int nova_cu_probe(nova_stream_t stream, uint32_t* out, int n_workgroups);

/* ------------------------------------------------------------------ kernel timing
 * When on, every kernel family launch inside the stage calls is bracketed by HIP events on
 * its stream.  nova_timing_read waits for the recorded events of `kind` (NOVA_KIND_*), returns
 * the summed GPU time and number of launches since the last read, and clears them. */
int nova_timing_enable(int on);
int nova_timing_read(int kind, double* total_ms, int* launches);

#ifdef __cplusplus
}
#endif
#endif /* NOVA_H */
