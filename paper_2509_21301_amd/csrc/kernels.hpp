// Host-side launchers of the gfx950 kernels (internal to libnova; the public C ABI is in nova.h).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

#ifndef NOVA_BF16_T
#define NOVA_BF16_T
typedef uint16_t bf16_t;
#endif

namespace nova {

enum Epi { EPI_STORE = 0, EPI_GELU = 1, EPI_RESID = 2, EPI_POS = 3, EPI_SWIGLU = 4, EPI_ARGMAX = 5 };

// C[M,N] = A[M,K] W[N,K]^T (+bias) with epilogue.  A has element type TA, row stride lda.
// STORE/GELU/SWIGLU write OT into out (row stride ldo); RESID adds into the fp32 out;
// POS writes fp32 out = acc + bias + pos[m % pos_rows] (pos is bf16 [pos_rows, N]).
struct GemmArgs {
  const void* A; int lda;
  const bf16_t* W; int ldw;
  int M, N, K;
  const bf16_t* bias;
  void* out; int ldo;
  const bf16_t* pos; int pos_rows;
  // optional split-K workspace: with too few output tiles to fill the GPU, the K range is cut
  // into up to 4 slices whose fp32 partial products land here ([slices][M][N]) and one more pass
  // sums them in slice order and applies the epilogue (STORE and RESID only)
  float* split_ws = nullptr; size_t split_ws_floats = 0;
  // set by the launcher, not by callers: K slice per workgroup and partial stride
  int kslice = 0; long split_stride = 0;
  // optional, STORE only: output columns from v_col0 on (the V of a fused QKV projection) go
  // transposed to vt instead of out: column v_col0 + h * vt_hd + d of row m = b * vt_tokens + t
  // lands at vt[((b * heads + h) * vt_hd + d) * vt_pad + t].  Requires v_col0 % 256 == 0,
  // vt_tokens % 8 == 0 and vt_pad % 8 == 0 (checked by the caller).
  void* vt = nullptr; int v_col0 = 0, vt_hd = 0, vt_tokens = 0, vt_pad = 0;
  int vt_row0 = 0;            // set by the launcher: row m of this launch is row vt_row0 + m above
  // bf16 only: always 128x128 tiles of 4 waves, unsplit (a kernel that leaves room on every CU for
  // another kernel's workgroups: the intra-CU co-residency variant)
  bool small_tiles = false;
  // RESID without bias only: when set and K is split, the K-slice partials are left in split_ws
  // ([slices][M][N]) for the caller to fold into out (split_norm_rows), and *slices_out gets the
  // slice count; otherwise *slices_out = 0 and out is complete
  int* slices_out = nullptr;
};
template <typename TA, typename OT>
hipError_t gemm(const GemmArgs& p, int epi, hipStream_t s);

// Thin GEMM for decode (M = B <= 32 rows): weights streamed once, split over K if needed.
// out gets epilogue epi (STORE: OT [B, ldo]; RESID: fp32 += ; SWIGLU: OT [B, N/2];
// ARGMAX: optional fp32 logits in out, greedy argmax merged into argmax_keys[b], which must be
// zero beforehand; argmax_finish() turns the keys into token ids).
// partial is fp32 workspace of gemv_partial_floats() floats laid out [split][B][N].  With
// gemv_splits() > 1 and out == null the partials are left for the caller's fused reduction.
struct GemvArgs {
  const void* X; int ldx;
  const bf16_t* W; int ldw;
  int B, N, K;
  void* out; int ldo;
  float* partial;
  unsigned long long* argmax_keys;
  // RMSNorm folded into its neighbours.  Consumer: when ss_in is set, X holds x * gain (the
  // residual times the norm's gain, written by the producer) and output column b is scaled by
  // rsqrt(sum_t ss_in[t * B + b] / K + eps) over t < ss_parts, the per-tile partial sums of
  // squares of row b of x (added in a fixed order, so results do not depend on scheduling).
  const float* ss_in = nullptr;
  int ss_parts = 0;
  float eps = 0.f;
  // Residual producer (EPI_RESID into fp32 out): ss_out[t * B + b] receives the sum of squares of
  // the updated row b over output tile t (64 rows of N), and when gain_out is set aout[b][n] =
  // x_new[b][n] * gain_out[n] in the activation type (row pitch ldao).  With split-K,
  // counters[N / 64] (zero on entry, zero again on exit) let the last split of each tile fold all
  // partials into out.
  float* ss_out = nullptr;
  unsigned* counters = nullptr;
  const bf16_t* gain_out = nullptr;
  void* aout = nullptr;
  int ldao = 0;
  // compute units the launch's stream may use (its CU partition, or the whole GPU): the K split
  // is chosen from it
  int cus = 0;
};
int gemv_splits(int N, int K, int B, bool f32x, int cus);
size_t gemv_partial_floats(int B, int N, int K, bool f32x, int cus);
template <typename TX, typename OT>
hipError_t gemv(const GemvArgs& p, int epi, hipStream_t s);

// Flash attention (bidirectional or causal, grouped-query) for encode and prefill.
// q, k: rows of the packed projection output; element (token t, head h, dim c) at
//   base + t * row_stride + h * D + c  (per-batch offset batch_stride).
// vt: V transposed, [batch][n_kv][D][sk_pad] (keys >= sk zero-filled up to sk_pad, a multiple of 64).
// out: [batch * sq, n_q * D] rows.
struct AttnArgs {
  const void* q; long q_row, q_batch;
  const void* k; long k_row, k_batch;
  const void* vt; int sk_pad;
  void* out; long o_row, o_batch;
  int sq, sk, n_q, n_kv, batch;
  int causal;
  // optional scratch (bidirectional bf16, head_dim <= 80): when the query blocks fill the GPU's
  // workgroup slots badly, the keys are cut into up to 3 ranges whose normalised partial outputs
  // (bf16) and (max, sum) land here, and a second pass merges them
  void* part = nullptr; size_t part_bytes = 0;
  int cus = 0;                // compute units of the stream (0: all 256)
  int kv_parts = 1;           // set by the launcher
  // optional (causal bf16): with part and counters ([batch * n_q][query blocks of 128], zero on
  // entry, zero again on return), the heaviest query blocks are cut into key ranges whose fp32
  // partials land in part; the last range of a block to finish merges them
  unsigned* counters = nullptr;
  int kv_tmax = 0, kv_units = 0, kv_slots = 0;   // set by the launcher
};
template <typename T>
hipError_t attention(const AttnArgs& p, int head_dim, hipStream_t s);

// Paged decode attention: one query per sequence against its paged KV blocks.
struct DecAttnArgs {
  const float* qkv;           // QKV projection, fp32 [qkv_splits][B][(n_q + 2 n_kv) D]: split-K slabs,
  int qkv_splits;             //   summed and rotated here (q and k at pos)
  const float* rope;          // [B][2][D/2]: sines, then cosines of each sequence's position
  void* kpool;                // [num_blocks, n_kv, block, D] for this layer; the step's k is appended
  void* vpool;                // [num_blocks, n_kv, D, block]; the step's v is appended
  const int* tables; int max_blocks;
  const int* pos;             // query position; context = pos + 1
  void* out;                  // [B, n_q * D]
  float* partial;             // workspace: split partials
  int B, n_q, n_kv, block, max_ctx;
};
size_t dec_attn_partial_floats(int B, int n_q, int D, int max_ctx, int n_kv);
template <typename T>
hipError_t decode_attention(const DecAttnArgs& p, int head_dim, hipStream_t s);

// Decode linear on the vector ALUs (no LDS, no matrix cores): out[B, ldo] += X[B, K] W[N, K]^T in
// fp32, B <= 4, K % 512 == 0.  The low-footprint decode kernel of the intra-CU co-residency variant.
hipError_t gemv_valu(const bf16_t* X, int ldx, const bf16_t* W, int ldw, int B, int N, int K, float* out, int ldo,
                     hipStream_t s);

// ---- small memory-bound kernels
// LayerNorm (ln=1, with shift b) or RMSNorm (ln=0) of fp32 rows into T rows.
// merge>1: row m = (img, py, px) of a (gh, gw) grid goes to merged row (img, py/m, px/m),
// column block (py%m)*m + px%m; out row stride is then merge*merge*H.
template <typename T>
hipError_t norm_rows(const float* x, int M, int H, const bf16_t* g, const bf16_t* b, float eps, int ln,
                     T* out, int ldo, int merge, int gh, int gw, hipStream_t s);
// The same norm after folding a K-split residual projection into x: x[m] += the sum of the
// `slices` fp32 partials part[k * pstride + m * H + n] in slice order (pstride >= M * H), written
// back, then the norm of the updated rows into out (merge 1).  The partials carry no bias.
template <typename T>
hipError_t split_norm_rows(const float* part, int slices, size_t pstride, float* x, int M, int H, const bf16_t* g,
                           const bf16_t* b, float eps, int ln, T* out, int ldo, hipStream_t s);
// Image [B, H, W, 3] bf16 -> patch rows [B*gh*gw, kpad] (zero padded), order (py, px, c).
template <typename T>
hipError_t patchify(const bf16_t* img, int B, int H, int W, int p, int kpad, T* out, hipStream_t s);
// Zero columns [c0, ld) of `rows` rows of pitch ld (the key padding of a V^T buffer).
template <typename T>
hipError_t zero_tail_cols(T* buf, long rows, int ld, int c0, hipStream_t s);
// Split a packed QKV projection.  Rotates q and k in place when rope_theta > 0 (positions
// pos0 + t), writes V transposed for attention (vt), and when tables != null writes the
// rotated K and V of every token into the paged cache.
// zero != null: also sets zero[0 .. nzero) to 0 (the attention's arrival counters).
template <typename T>
hipError_t qkv_prefill(T* qkv, int S, int batch, int n_q, int n_kv, int D, float rope_theta, int pos0,
                       T* vt, int sk_pad, T* kpool, T* vpool, const int* table, int block, hipStream_t s,
                       unsigned* zero = nullptr, int nzero = 0);
// Decode residual + RMSNorm, one workgroup per row: x[b] += sum_s partial[s][b] (if splits > 0),
// then a[b] = x[b] / sqrt(mean(x[b]^2) + eps) * g.
// keys != null: also zero keys[b] for the fused argmax of the projection that follows.
template <typename T>
hipError_t resid_rmsnorm(const float* partial, int splits, float* x, int B, int H, const bf16_t* g, float eps, T* a,
                         int lda, unsigned long long* keys, hipStream_t s);
// Decode residual fold, column tiles of 64 over the whole GPU (H % 64 == 0): x[b] += sum_s
// partial[s][b] (if splits > 0), a[b] = x[b] * g, ss_out[t * B + b] = sum of squares of tile t of
// x[b], for a consumer that normalises from the H / 64 tile parts.
template <typename T>
hipError_t resid_fold(const float* partial, int splits, float* x, int B, int H, const bf16_t* g, T* a, int lda,
                      float* ss_out, hipStream_t s);
// ids[b] = the token id packed in keys[b] by the fused argmax.
hipError_t argmax_finish(const unsigned long long* keys, int B, int* ids, hipStream_t s);
// x[r] = r < n_vis ? vis[r] : embed[ids[r - n_vis]]  (fp32 out)
// Decode step start: x[b] = embed[ids[b]] (fp32), a[b] = x[b] * g in the activation type;
// ss0[0 * B + b] = sum of squares of x[b] and ss0[t * B + b] = 0 for 0 < t < ss_parts; zeroes
// keys[B] and counters[n_counters]; rope[b] = the rotary sines then cosines of position pos[b]
// (2 x D/2 floats), which every layer's decode attention reads.
template <typename T>
hipError_t decode_embed(const int* ids, int B, const bf16_t* embed, int H, const bf16_t* g, float* x, T* a, float* ss0,
                        int ss_parts, unsigned long long* keys, unsigned* counters, int n_counters, const int* pos,
                        float theta, int D, float* rope, hipStream_t s);
template <typename T>
hipError_t embed_rows(const T* vis, int n_vis, const int* ids, int n_ids, const bf16_t* embed, int H, float* x,
                      hipStream_t s);
hipError_t argmax_rows(const float* logits, int B, int V, int* out, hipStream_t s);
hipError_t cu_probe(hipStream_t s, uint32_t* out, int n);

}  // namespace nova
