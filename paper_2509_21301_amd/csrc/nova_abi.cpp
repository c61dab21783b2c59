// libnova C ABI: weight layouts, model handles, the three stage calls, CU partitions, layer
// prefetch and kernel timing.  Stage calls only enqueue kernels on the caller's stream; they
// allocate no device memory (workspaces come from the caller).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/nova.h"
#include "kernels.hpp"

using nova::GemmArgs;
using nova::GemvArgs;

// ------------------------------------------------------------------ errors
static thread_local std::string t_err;

static int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  t_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                                    \
  do {                                                                                                   \
    hipError_t e_ = (expr);                                                                              \
    if (e_ != hipSuccess) return fail(NOVA_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));         \
  } while (0)

extern "C" const char* nova_last_error(void) { return t_err.c_str(); }

// ------------------------------------------------------------------ global state
namespace {
struct Global {
  int device = -1;
  int cus = 0;
  std::mutex mu;
  std::map<std::vector<uint32_t>, hipStream_t> mask_streams;   // partition stream pool
  std::map<std::vector<uint32_t>, uint64_t> mask_used;          // its last use (a counter)
  uint64_t uses = 0;
  hipStream_t full_streams[3] = {nullptr, nullptr, nullptr};   // whole-GPU mask, one per stage
  hipStream_t stage_stream[3] = {nullptr, nullptr, nullptr};
  hipEvent_t stage_switch[3] = {nullptr, nullptr, nullptr};
  // timing
  bool timing = false;
  std::vector<hipEvent_t> ev_free;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev_used[NOVA_KIND_MISC + 1];
};
Global g;

// Compute units a stream may use: its CU mask's when it is one of the partition streams, else the
// whole GPU's.
int stream_cus(hipStream_t s) {
  std::lock_guard<std::mutex> lk(g.mu);
  for (const auto& ms : g.mask_streams)
    if (ms.second == s) {
      int n = 0;
      for (uint32_t w : ms.first) n += __builtin_popcount(w);
      return n > 0 ? n : g.cus;
    }
  return g.cus;
}

hipEvent_t take_event() {
  std::lock_guard<std::mutex> lk(g.mu);
  if (!g.ev_free.empty()) {
    hipEvent_t e = g.ev_free.back();
    g.ev_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Run one kernel-family launch, bracketed by timing events when timing is on.
template <typename F>
int timed(int kind, hipStream_t s, const char* what, F&& f) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (g.timing) {
    e0 = take_event();
    if (e0) hipEventRecord(e0, s);
  }
  hipError_t err = f();
  if (err != hipSuccess) return fail(NOVA_EHIP, "%s launch failed: %s", what, hipGetErrorString(err));
  if (g.timing && e0) {
    e1 = take_event();
    if (e1) {
      hipEventRecord(e1, s);
      std::lock_guard<std::mutex> lk(g.mu);
      g.ev_used[kind].push_back({e0, e1});
    }
  }
  return NOVA_OK;
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline int round_up(int x, int m) { return (x + m - 1) / m * m; }
inline bool aligned(const void* p) { return ((uintptr_t)p & 255) == 0; }
}  // namespace

#define CALL(kind, stream, expr)                                                   \
  do {                                                                             \
    int rc_ = timed(kind, stream, #expr, [&]() { return (expr); });               \
    if (rc_ != NOVA_OK) return rc_;                                                \
  } while (0)

namespace {
int scratch_for_current_device(void** out);
}

extern "C" int nova_init(int device) {
  int n = 0;
  HIP_TRY(hipGetDeviceCount(&n));
  if (device < 0 || device >= n) return fail(NOVA_EINVAL, "device %d out of range (%d devices)", device, n);
  HIP_TRY(hipSetDevice(device));
  hipDeviceProp_t prop;
  HIP_TRY(hipGetDeviceProperties(&prop, device));
  g.device = device;
  g.cus = prop.multiProcessorCount;
  void* scr = nullptr;   // the allocation-free decode's scratch address on this device
  return scratch_for_current_device(&scr);
}

extern "C" void nova_shutdown(void) {
  std::lock_guard<std::mutex> lk(g.mu);
  for (auto& kv : g.mask_streams) hipStreamDestroy(kv.second);
  g.mask_used.clear();
  for (auto& fs : g.full_streams) {
    if (fs) hipStreamDestroy(fs);
    fs = nullptr;
  }
  g.mask_streams.clear();
  for (int i = 0; i < 3; ++i) {
    if (g.stage_switch[i]) hipEventDestroy(g.stage_switch[i]);
    g.stage_switch[i] = nullptr;
    g.stage_stream[i] = nullptr;
  }
  for (auto e : g.ev_free) hipEventDestroy(e);
  g.ev_free.clear();
  for (auto& v : g.ev_used) {
    for (auto& pr : v) { hipEventDestroy(pr.first); hipEventDestroy(pr.second); }
    v.clear();
  }
  g.timing = false;
}

extern "C" int nova_device_cus(void) { return g.cus; }

// ------------------------------------------------------------------ layouts
namespace {
struct Layout {
  std::vector<size_t> off;
  size_t bytes = 0;
  void add(size_t elems) {
    off.push_back(bytes);
    bytes = align256(bytes + elems * 2);
  }
};
int vit_kpad(const nova_vit_config& c) { return round_up(3 * c.patch * c.patch, 64); }
int vit_ip(const nova_vit_config& c) { return round_up(c.mlp, 256); }
int vit_npatch(const nova_vit_config& c) { return (c.image_h / c.patch) * (c.image_w / c.patch); }
int llm_ip(const nova_llm_config& c) { return round_up(c.inter, 256); }

int check_vit_cfg(const nova_vit_config* c) {
  if (!c) return fail(NOVA_EINVAL, "null vit config");
  if (c->hidden <= 0 || c->heads <= 0 || c->hidden % c->heads || c->mlp <= 0 || c->layers < 0 || c->patch <= 0 ||
      c->out_hidden <= 0 || c->image_h <= 0 || c->image_w <= 0)
    return fail(NOVA_EINVAL, "vit config: non-positive or inconsistent sizes");
  if (c->merge != 1 && c->merge != 2) return fail(NOVA_EUNSUPPORTED, "vit merge must be 1 or 2");
  if (c->image_h % (c->patch * c->merge) || c->image_w % (c->patch * c->merge))
    return fail(NOVA_EINVAL, "image size must be a multiple of patch*merge");
  const int d = c->hidden / c->heads;
  if (d != 64 && d != 80 && d != 128) return fail(NOVA_EUNSUPPORTED, "vit head_dim %d (supported: 64, 80, 128)", d);
  if (c->act == NOVA_ACT_F32 && d > 80) return fail(NOVA_EUNSUPPORTED, "fp32 mode supports head_dim <= 80");
  if (c->hidden % 128 || c->out_hidden % 128) return fail(NOVA_EUNSUPPORTED, "vit hidden and out_hidden must be multiples of 128");
  if (c->act != NOVA_ACT_BF16 && c->act != NOVA_ACT_F32) return fail(NOVA_EINVAL, "act must be NOVA_ACT_BF16 or NOVA_ACT_F32");
  return NOVA_OK;
}

int check_llm_cfg(const nova_llm_config* c) {
  if (!c) return fail(NOVA_EINVAL, "null llm config");
  if (c->hidden <= 0 || c->n_q <= 0 || c->n_kv <= 0 || c->n_q % c->n_kv || c->inter <= 0 || c->vocab <= 0 ||
      c->layers < 0)
    return fail(NOVA_EINVAL, "llm config: non-positive or inconsistent sizes");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(NOVA_EUNSUPPORTED, "llm head_dim %d (supported: 64, 128)", c->head_dim);
  if (c->act == NOVA_ACT_F32 && c->head_dim > 80) return fail(NOVA_EUNSUPPORTED, "fp32 mode supports head_dim <= 80");
  if (c->block != 16) return fail(NOVA_EUNSUPPORTED, "KV block must be 16 tokens");
  if (c->n_q / c->n_kv > 16) return fail(NOVA_EUNSUPPORTED, "at most 16 query heads per KV head");
  if (c->hidden % 256 || (c->n_q * c->head_dim) % 256 || c->vocab % 128)
    return fail(NOVA_EUNSUPPORTED, "hidden and n_q*head_dim must be multiples of 256, vocab of 128");
  if (c->hidden > 4096) return fail(NOVA_EUNSUPPORTED, "hidden %d above 4096 (decode normalises from at most 64 column tiles)", c->hidden);
  if (((c->n_q + 2 * c->n_kv) * c->head_dim) % 128) return fail(NOVA_EUNSUPPORTED, "(n_q+2n_kv)*head_dim must be a multiple of 128");
  if (!(c->rope_theta > 0.f)) return fail(NOVA_EINVAL, "rope_theta must be positive");
  if (c->act != NOVA_ACT_BF16 && c->act != NOVA_ACT_F32) return fail(NOVA_EINVAL, "act must be NOVA_ACT_BF16 or NOVA_ACT_F32");
  return NOVA_OK;
}

Layout vit_embed_layout(const nova_vit_config& c) {
  Layout l;
  l.add((size_t)c.hidden * vit_kpad(c));
  l.add(c.hidden);
  l.add((size_t)vit_npatch(c) * c.hidden);
  return l;
}
Layout vit_layer_layout(const nova_vit_config& c) {
  const size_t H = c.hidden, I = vit_ip(c);
  Layout l;
  l.add(H); l.add(H);
  l.add(3 * H * H); l.add(3 * H);
  l.add(H * H); l.add(H);
  l.add(H); l.add(H);
  l.add(I * H); l.add(I);
  l.add(H * I); l.add(H);
  return l;
}
Layout vit_head_layout(const nova_vit_config& c) {
  Layout l;
  l.add(c.hidden); l.add(c.hidden);
  l.add((size_t)c.out_hidden * c.merge * c.merge * c.hidden);
  l.add(c.out_hidden);
  return l;
}
Layout llm_layer_layout(const nova_llm_config& c) {
  const size_t H = c.hidden, I = llm_ip(c), d = c.head_dim;
  Layout l;
  l.add(H);
  l.add((c.n_q + 2 * c.n_kv) * d * H);
  l.add(H * c.n_q * d);
  l.add(H);
  l.add(2 * I * H);
  l.add(H * I);
  return l;
}
Layout llm_head_layout(const nova_llm_config& c) {
  Layout l;
  l.add(c.hidden);
  l.add((size_t)c.vocab * c.hidden);
  return l;
}
int emit(const Layout& l, size_t* offsets, size_t* bytes) {
  if (offsets)
    for (size_t i = 0; i < l.off.size(); ++i) offsets[i] = l.off[i];
  if (bytes) *bytes = l.bytes;
  return NOVA_OK;
}
}  // namespace

extern "C" int nova_vit_embed_layout(const nova_vit_config* c, size_t* o, size_t* b) {
  int rc = check_vit_cfg(c);
  return rc ? rc : emit(vit_embed_layout(*c), o, b);
}
extern "C" int nova_vit_layer_layout(const nova_vit_config* c, size_t* o, size_t* b) {
  int rc = check_vit_cfg(c);
  return rc ? rc : emit(vit_layer_layout(*c), o, b);
}
extern "C" int nova_vit_head_layout(const nova_vit_config* c, size_t* o, size_t* b) {
  int rc = check_vit_cfg(c);
  return rc ? rc : emit(vit_head_layout(*c), o, b);
}
extern "C" int nova_llm_layer_layout(const nova_llm_config* c, size_t* o, size_t* b) {
  int rc = check_llm_cfg(c);
  return rc ? rc : emit(llm_layer_layout(*c), o, b);
}
extern "C" int nova_llm_head_layout(const nova_llm_config* c, size_t* o, size_t* b) {
  int rc = check_llm_cfg(c);
  return rc ? rc : emit(llm_head_layout(*c), o, b);
}

// ------------------------------------------------------------------ workspace carving
namespace {
struct Carve {
  char* base;
  size_t used = 0;
  explicit Carve(void* b) : base((char*)b) {}
  template <typename T>
  T* take(size_t elems) {
    T* p = base ? (T*)(base + used) : nullptr;
    used = align256(used + elems * sizeof(T));
    return p;
  }
};
}  // namespace

// ------------------------------------------------------------------ vision encoder
struct nova_vit {
  nova_vit_desc d;
  Layout emb, lay, head;
  int kpad, ip, npatch, nout, hd;
  bool offload = false;
  hipStream_t copy_stream = nullptr;
  std::vector<hipEvent_t> ready, freed;
  std::vector<int> slot_layer;            // logical layer each physical slot holds (or is receiving), -1 if none
  std::vector<char> freed_recorded;
  unsigned long long copies = 0;          // host-to-device layer copies issued so far
};

namespace {
int find_slot(const nova_vit* v, int layer) {
  for (int p = 0; p < (int)v->slot_layer.size(); ++p)
    if (v->slot_layer[p] == layer) return p;
  return -1;
}

// Copy logical layer `layer` into physical slot p on stream cs, once the last compute use of p
// has finished; the slot's ready event then marks the copy done.
int copy_into_slot(nova_vit* v, int layer, int p, hipStream_t cs) {
  if (v->freed_recorded[p]) HIP_TRY(hipStreamWaitEvent(cs, v->freed[p], 0));
  const size_t lb = v->lay.bytes;
  HIP_TRY(hipMemcpyAsync((char*)v->d.slots + (size_t)p * lb, (const char*)v->d.host_layers + (size_t)layer * lb, lb,
                         hipMemcpyHostToDevice, cs));
  HIP_TRY(hipEventRecord(v->ready[p], cs));
  v->slot_layer[p] = layer;
  ++v->copies;
  return NOVA_OK;
}
}  // namespace

extern "C" int nova_vit_create(const nova_vit_desc* desc, nova_vit** out) {
  if (!desc || !out) return fail(NOVA_EINVAL, "null argument");
  int rc = check_vit_cfg(&desc->cfg);
  if (rc) return rc;
  const nova_vit_config& c = desc->cfg;
  if (!desc->embed || !desc->head || !aligned(desc->embed) || !aligned(desc->head))
    return fail(NOVA_EINVAL, "embed/head blobs must be non-null and 256-byte aligned");
  const bool off = desc->host_layers != nullptr;
  if (off) {
    if (!desc->slots || !aligned(desc->slots)) return fail(NOVA_EINVAL, "offload needs 256-byte aligned device slots");
    if (desc->n_slots < 2 || desc->n_slots >= c.layers) return fail(NOVA_EINVAL, "offload needs 2 <= n_slots < layers");
  } else if (c.layers > 0 && (!desc->layers || !aligned(desc->layers))) {
    return fail(NOVA_EINVAL, "resident layers must be non-null and 256-byte aligned");
  }
  nova_vit* v = new nova_vit();
  v->d = *desc;
  v->emb = vit_embed_layout(c);
  v->lay = vit_layer_layout(c);
  v->head = vit_head_layout(c);
  v->kpad = vit_kpad(c);
  v->ip = vit_ip(c);
  v->npatch = vit_npatch(c);
  v->nout = v->npatch / (c.merge * c.merge);
  v->hd = c.hidden / c.heads;
  v->offload = off;
  if (off) {
    const int K = desc->n_slots;
    v->ready.assign(K, nullptr);
    v->freed.assign(K, nullptr);
    v->slot_layer.assign(K, -1);
    v->freed_recorded.assign(K, 0);
    hipError_t e = hipStreamCreateWithFlags(&v->copy_stream, hipStreamNonBlocking);
    for (int i = 0; e == hipSuccess && i < K; ++i) {
      e = hipEventCreateWithFlags(&v->ready[i], hipEventDisableTiming);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&v->freed[i], hipEventDisableTiming);
    }
    if (e != hipSuccess) {
      nova_vit_destroy(v);
      return fail(NOVA_EHIP, "creating offload stream/events: %s", hipGetErrorString(e));
    }
  }
  *out = v;
  return NOVA_OK;
}

extern "C" void nova_vit_destroy(nova_vit* v) {
  if (!v) return;
  if (v->copy_stream) { hipStreamSynchronize(v->copy_stream); hipStreamDestroy(v->copy_stream); }
  for (auto e : v->ready) if (e) hipEventDestroy(e);
  for (auto e : v->freed) if (e) hipEventDestroy(e);
  delete v;
}

namespace {
template <typename T>
size_t vit_ws(const nova_vit* v, int B, Carve* cv) {
  const nova_vit_config& c = v->d.cfg;
  const size_t M = (size_t)B * v->npatch, H = c.hidden;
  const int skp = round_up(v->npatch, 64);
  Carve tmp(nullptr);
  Carve& w = cv ? *cv : tmp;
  w.take<T>(M * v->kpad);           // patches
  w.take<float>(M * H);             // residual stream
  w.take<T>(M * H);                 // normed rows
  w.take<T>(M * 3 * H);             // qkv (also the merged rows of the adapter)
  w.take<T>((size_t)B * H * skp);   // V^T
  w.take<T>(M * H);                 // attention output
  w.take<T>(M * v->ip);             // MLP hidden
  return w.used;
}
}  // namespace

extern "C" size_t nova_vit_workspace_bytes(const nova_vit* v, int batch) {
  if (!v || batch <= 0) return 0;
  return v->d.cfg.act == NOVA_ACT_F32 ? vit_ws<float>(v, batch, nullptr) : vit_ws<bf16_t>(v, batch, nullptr);
}

extern "C" int nova_prefetch_layer(nova_vit* v, int layer, nova_stream_t cs_in) {
  if (!v) return fail(NOVA_EINVAL, "null vit");
  if (!v->offload) return fail(NOVA_EINVAL, "model has no layer offload");
  if (layer < 0 || layer >= v->d.cfg.layers) return fail(NOVA_EINVAL, "layer %d out of range", layer);
  hipStream_t cs = cs_in ? (hipStream_t)cs_in : v->copy_stream;
  if (find_slot(v, layer) >= 0) return NOVA_OK;        // already resident (or in flight)
  // the slot Eq. 7 gives it: the one that holds layer - K; else an empty one; else slot layer mod K
  const int K = v->d.n_slots, L = v->d.cfg.layers;
  int p = find_slot(v, ((layer - K) % L + L) % L);
  if (p < 0) p = find_slot(v, -1);
  if (p < 0) p = layer % K;
  return copy_into_slot(v, layer, p, cs);
}

extern "C" int nova_vit_offload_state(const nova_vit* v, int* slot_layer, unsigned long long* copies) {
  if (!v) return fail(NOVA_EINVAL, "null vit");
  if (!v->offload) return fail(NOVA_EINVAL, "model has no layer offload");
  if (slot_layer)
    for (int p = 0; p < v->d.n_slots; ++p) slot_layer[p] = v->slot_layer[p];
  if (copies) *copies = v->copies;
  return NOVA_OK;
}

namespace {
template <typename T>
int vit_encode_t(nova_vit* v, const void* pixels, int B, void* out, void* ws, hipStream_t s) {
  const nova_vit_config& c = v->d.cfg;
  const int H = c.hidden, N = v->npatch, M = B * N, hd = v->hd, heads = c.heads;
  const int gh = c.image_h / c.patch, gw = c.image_w / c.patch;
  const int skp = round_up(N, 64);
  Carve w(ws);
  T* patches = w.take<T>((size_t)M * v->kpad);
  float* x = w.take<float>((size_t)M * H);
  T* a = w.take<T>((size_t)M * H);
  T* qkv = w.take<T>((size_t)M * 3 * H);
  T* vt = w.take<T>((size_t)B * H * skp);
  T* att = w.take<T>((size_t)M * H);
  T* hmlp = w.take<T>((size_t)M * v->ip);

  const char* emb = (const char*)v->d.embed;
  auto ew = [&](int i) { return (const bf16_t*)(emb + v->emb.off[i]); };
  CALL(NOVA_KIND_MISC, s, nova::patchify<T>((const bf16_t*)pixels, B, c.image_h, c.image_w, c.patch, v->kpad, patches, s));
  {
    GemmArgs p{patches, v->kpad, ew(0), v->kpad, M, H, v->kpad, ew(1), x, H, ew(2), N};
    CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_POS, s)));
  }
  const int L = c.layers, K = v->offload ? v->d.n_slots : 0;
  // the QKV projection writes V^T itself when V starts on a 256-column tile and tokens come in
  // eights; the keys past N then stay zero for the whole pass
  const bool vt_fused = (2 * H) % 256 == 0 && N % 8 == 0;
  if (vt_fused) CALL(NOVA_KIND_MISC, s, nova::zero_tail_cols<T>(vt, (long)B * H, skp, N, s));
  // the first K layers: already in their slots after an earlier call (its tail loaded them), else
  // all K copies are queued here at once rather than one per layer
  for (int l = 0; l < K; ++l)
    if (int rc = nova_prefetch_layer(v, l, nullptr)) return rc;
  for (int l = 0; l < L; ++l) {
    const char* lw;
    int slot = -1;
    if (v->offload) {
      slot = find_slot(v, l);
      if (slot < 0) {
        if (int rc = nova_prefetch_layer(v, l, nullptr)) return rc;
        slot = find_slot(v, l);
      }
      HIP_TRY(hipStreamWaitEvent(s, v->ready[slot], 0));
      lw = (const char*)v->d.slots + (size_t)slot * v->lay.bytes;
    } else {
      lw = (const char*)v->d.layers + (size_t)l * v->lay.bytes;
    }
    auto W = [&](int i) { return (const bf16_t*)(lw + v->lay.off[i]); };
    CALL(NOVA_KIND_MISC, s, nova::norm_rows<T>(x, M, H, W(0), W(1), c.eps, 1, a, H, 1, 0, 0, s));
    {
      GemmArgs p{a, H, W(2), H, M, 3 * H, H, W(3), qkv, 3 * H, nullptr, 0};
      if (vt_fused) {      // V straight to V^T from the projection's epilogue
        p.vt = vt, p.v_col0 = 2 * H, p.vt_hd = hd, p.vt_tokens = N, p.vt_pad = skp;
      }
      CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_STORE, s)));
    }
    if (!vt_fused)
      CALL(NOVA_KIND_MISC, s, nova::qkv_prefill<T>(qkv, N, B, heads, heads, hd, 0.f, 0, vt, skp, nullptr, nullptr, nullptr, 16, s));
    {
      nova::AttnArgs p{qkv, 3L * H, (long)N * 3 * H, qkv + H, 3L * H, (long)N * 3 * H, vt, skp, att, H, (long)N * H,
                       N, N, heads, heads, B, 0};
      p.part = hmlp, p.part_bytes = (size_t)M * v->ip * sizeof(T);      // the MLP hidden is free here
      p.cus = stream_cus(s);
      CALL(NOVA_KIND_ATTN, s, nova::attention<T>(p, hd, s));
    }
    {
      GemmArgs p{att, H, W(4), H, M, H, H, W(5), x, H, nullptr, 0};
      // K-slice partials, where the GEMM takes them: the MLP hidden is free here
      p.split_ws = reinterpret_cast<float*>(hmlp), p.split_ws_floats = (size_t)M * v->ip * sizeof(T) / sizeof(float);
      CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_RESID, s)));
    }
    CALL(NOVA_KIND_MISC, s, nova::norm_rows<T>(x, M, H, W(6), W(7), c.eps, 1, a, H, 1, 0, 0, s));
    {
      GemmArgs p{a, H, W(8), H, M, v->ip, H, W(9), hmlp, v->ip, nullptr, 0};
      CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_GELU, s)));
    }
    {
      GemmArgs p{hmlp, v->ip, W(10), v->ip, M, H, v->ip, W(11), x, H, nullptr, 0};
      // K-slice partials in the packed QKV buffer, free until the next layer's projection
      p.split_ws = reinterpret_cast<float*>(qkv), p.split_ws_floats = (size_t)M * 3 * H * sizeof(T) / sizeof(float);
      CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_RESID, s)));
    }
    if (v->offload) {
      // Eq. 7: the slot that held layer l receives layer (l + K) mod L once l's kernels are done
      HIP_TRY(hipEventRecord(v->freed[slot], s));
      v->freed_recorded[slot] = 1;
      const int nxt = (l + K) % L;
      if (find_slot(v, nxt) < 0)
        if (int rc = copy_into_slot(v, nxt, slot, v->copy_stream)) return rc;
    }
  }
  // adapter: LN per patch scattered into merged rows, then one Linear
  const char* hw = (const char*)v->d.head;
  auto HW = [&](int i) { return (const bf16_t*)(hw + v->head.off[i]); };
  const int m2 = c.merge * c.merge, Mo = B * v->nout;
  T* merged = qkv;   // [Mo, m2*H] fits in the qkv buffer
  CALL(NOVA_KIND_MISC, s, nova::norm_rows<T>(x, M, H, HW(0), HW(1), c.eps, 1, merged, m2 * H, c.merge, gh, gw, s));
  {
    GemmArgs p{merged, m2 * H, HW(2), m2 * H, Mo, c.out_hidden, m2 * H, HW(3), out, c.out_hidden, nullptr, 0};
    p.split_ws = reinterpret_cast<float*>(hmlp), p.split_ws_floats = (size_t)M * v->ip * sizeof(T) / sizeof(float);
    CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_STORE, s)));
  }
  return NOVA_OK;
}
}  // namespace

extern "C" int nova_vit_encode(nova_vit* v, const void* pixels, int batch, void* out, void* ws, size_t ws_bytes,
                               nova_stream_t stream) {
  if (!v) return fail(NOVA_EINVAL, "null vit");
  if (batch <= 0) return fail(NOVA_EINVAL, "batch must be positive");
  if (!pixels || !out || !ws || !aligned(pixels) || !aligned(out) || !aligned(ws))
    return fail(NOVA_EINVAL, "pixels/out/ws must be non-null and 256-byte aligned");
  const size_t need = nova_vit_workspace_bytes(v, batch);
  if (ws_bytes < need) return fail(NOVA_ENOSPACE, "workspace %zu < required %zu bytes", ws_bytes, need);
  hipStream_t s = (hipStream_t)stream;
  return v->d.cfg.act == NOVA_ACT_F32 ? vit_encode_t<float>(v, pixels, batch, out, ws, s)
                                      : vit_encode_t<bf16_t>(v, pixels, batch, out, ws, s);
}

// ------------------------------------------------------------------ LLM
struct nova_llm {
  nova_llm_desc d;
  Layout lay, head;
  int ip, qkvw;
};

extern "C" int nova_llm_create(const nova_llm_desc* desc, nova_llm** out) {
  if (!desc || !out) return fail(NOVA_EINVAL, "null argument");
  int rc = check_llm_cfg(&desc->cfg);
  if (rc) return rc;
  if (!desc->embed || !desc->head || !aligned(desc->embed) || !aligned(desc->head) ||
      (desc->cfg.layers > 0 && (!desc->layers || !aligned(desc->layers))))
    return fail(NOVA_EINVAL, "embed/layers/head must be non-null and 256-byte aligned");
  nova_llm* m = new nova_llm();
  m->d = *desc;
  m->lay = llm_layer_layout(desc->cfg);
  m->head = llm_head_layout(desc->cfg);
  m->ip = llm_ip(desc->cfg);
  m->qkvw = (desc->cfg.n_q + 2 * desc->cfg.n_kv) * desc->cfg.head_dim;
  *out = m;
  return NOVA_OK;
}

extern "C" void nova_llm_destroy(nova_llm* m) { delete m; }

extern "C" size_t nova_kv_bytes(const nova_llm* m, int num_blocks) {
  if (!m || num_blocks <= 0) return 0;
  const nova_llm_config& c = m->d.cfg;
  const size_t el = c.act == NOVA_ACT_F32 ? 4 : 2;
  return (size_t)c.layers * num_blocks * c.n_kv * c.block * c.head_dim * el;
}

namespace {
// Split-K partials of the prefill projections: up to 4 K slices of the widest split output.
size_t prefill_split_floats(const nova_llm* m, int S) {
  return (size_t)4 * S * std::max<size_t>(m->d.cfg.hidden, m->qkvw);
}

template <typename T>
size_t prefill_ws(const nova_llm* m, int S, Carve* cv) {
  const nova_llm_config& c = m->d.cfg;
  Carve tmp(nullptr);
  Carve& w = cv ? *cv : tmp;
  const size_t H = c.hidden;
  w.take<float>((size_t)S * H);                                  // residual
  w.take<T>((size_t)S * H);                                      // normed
  w.take<T>((size_t)S * m->qkvw);                                // qkv
  w.take<T>((size_t)c.n_kv * c.head_dim * round_up(S, 64));      // V^T
  w.take<T>((size_t)S * c.n_q * c.head_dim);                     // attention out
  w.take<T>((size_t)S * m->ip);                                  // MLP hidden
  w.take<unsigned long long>(1);                                 // argmax key
  w.take<float>(prefill_split_floats(m, S));                     // split-K partials
  w.take<unsigned>((size_t)c.n_q * ((S + 127) / 128));           // attention arrival counters
  return w.used;
}
template <typename T>
struct DecodeBufs {
  float* x;                   // residual stream [B][H]
  T* a;                       // x times the next RMSNorm's gain, input of the next projection [B][H]
  float* qkv;                 // QKV projection (fp32) when not split
  T* att;                     // attention output
  T* hm;                      // MLP hidden
  unsigned long long* keys;   // greedy argmax keys
  float* ss;                  // per-tile row sums of squares of the 2 L + 1 fused RMSNorms [2L+1][H/64][B]
  unsigned* counters;         // split-K arrival counters of the O and down projections [2L][H/64]
  float* rope;                // rotary sines and cosines of each sequence's position [B][2][D/2]
  float* part;                // split-K partials
  float* apart;               // decode-attention split partials
  size_t used;
};

// The decode step's workspace, carved from base (sizes only when base is null).
template <typename T>
DecodeBufs<T> decode_bufs(const nova_llm* m, int B, int max_ctx, void* base) {
  const nova_llm_config& c = m->d.cfg;
  Carve w(base);
  DecodeBufs<T> d;
  const size_t H = c.hidden;
  const int qd = c.n_q * c.head_dim;
  d.x = w.take<float>((size_t)B * H);
  d.a = w.take<T>((size_t)B * H);
  d.qkv = w.take<float>((size_t)B * m->qkvw);
  d.att = w.take<T>((size_t)B * qd);
  d.hm = w.take<T>((size_t)B * m->ip);
  d.keys = w.take<unsigned long long>((size_t)B);
  d.ss = w.take<float>((size_t)(2 * c.layers + 1) * (H / 64) * B);
  d.counters = w.take<unsigned>((size_t)2 * c.layers * (H / 64));
  d.rope = w.take<float>((size_t)B * c.head_dim);
  size_t part = 0;
  const bool f32 = sizeof(T) == 4;
  part = std::max(part, nova::gemv_partial_floats(B, m->qkvw, c.hidden, f32, g.cus));
  part = std::max(part, nova::gemv_partial_floats(B, c.hidden, qd, f32, g.cus));
  part = std::max(part, nova::gemv_partial_floats(B, 2 * m->ip, c.hidden, f32, g.cus));
  part = std::max(part, nova::gemv_partial_floats(B, c.hidden, m->ip, f32, g.cus));
  part = std::max(part, nova::gemv_partial_floats(B, c.vocab, c.hidden, f32, g.cus));
  d.part = w.take<float>(part);
  d.apart = w.take<float>(nova::dec_attn_partial_floats(B, c.n_q, c.head_dim, max_ctx, c.n_kv));
  d.used = w.used;
  return d;
}
}  // namespace

extern "C" size_t nova_llm_prefill_workspace_bytes(const nova_llm* m, int seq) {
  if (!m || seq <= 0) return 0;
  return m->d.cfg.act == NOVA_ACT_F32 ? prefill_ws<float>(m, seq, nullptr) : prefill_ws<bf16_t>(m, seq, nullptr);
}
extern "C" size_t nova_llm_decode_workspace_bytes(const nova_llm* m, int batch, int max_ctx) {
  if (!m || batch <= 0 || max_ctx <= 0) return 0;
  return m->d.cfg.act == NOVA_ACT_F32 ? decode_bufs<float>(m, batch, max_ctx, nullptr).used
                                      : decode_bufs<bf16_t>(m, batch, max_ctx, nullptr).used;
}

namespace {
template <typename T>
int llm_prefill_t(const nova_llm* m, const T* vis, int n_vis, const int* ids, int n_text, const int* table,
                  const nova_kv* kv, int* next_id, float* logits_out, void* ws, hipStream_t s) {
  const nova_llm_config& c = m->d.cfg;
  const int S = n_vis + n_text, H = c.hidden, D = c.head_dim, qd = c.n_q * D;
  const int skp = round_up(S, 64);
  Carve w(ws);
  float* x = w.take<float>((size_t)S * H);
  T* a = w.take<T>((size_t)S * H);
  T* qkv = w.take<T>((size_t)S * m->qkvw);
  T* vt = w.take<T>((size_t)c.n_kv * D * skp);
  T* att = w.take<T>((size_t)S * qd);
  T* hm = w.take<T>((size_t)S * m->ip);
  unsigned long long* keys = w.take<unsigned long long>(1);
  const size_t split_floats = prefill_split_floats(m, S);
  float* split_ws = w.take<float>(split_floats);
  const int n_cnt = c.n_q * ((S + 127) / 128);
  unsigned* att_cnt = w.take<unsigned>((size_t)n_cnt);
  const size_t kv_layer = (size_t)kv->num_blocks * c.n_kv * c.block * D;
  const int cus = stream_cus(s);
  // the QKV, O and down projections may split K when their tiles cannot fill the GPU
  auto with_split = [&](GemmArgs p) {
    p.split_ws = split_ws;
    p.split_ws_floats = split_floats;
    return p;
  };

  CALL(NOVA_KIND_MISC, s, nova::embed_rows<T>(vis, n_vis, ids, n_text, (const bf16_t*)m->d.embed, H, x, s));
  // a residual projection (O, down) whose K is split leaves its slices for the RMSNorm that reads
  // x next to fold in (one pass over x instead of a reduction pass and a norm pass)
  auto resid_then_norm = [&](const GemmArgs& g, const bf16_t* gain) -> int {
    GemmArgs p = g;
    int slices = 0;
    p.slices_out = &slices;
    CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_RESID, s)));
    if (slices > 0)
      CALL(NOVA_KIND_MISC, s, nova::split_norm_rows<T>(split_ws, slices, (size_t)S * H, x, S, H, gain, nullptr, c.eps, 0, a, H, s));
    else
      CALL(NOVA_KIND_MISC, s, nova::norm_rows<T>(x, S, H, gain, nullptr, c.eps, 0, a, H, 1, 0, 0, s));
    return (int)NOVA_OK;
  };
  for (int l = 0; l < c.layers; ++l) {
    const char* lw = (const char*)m->d.layers + (size_t)l * m->lay.bytes;
    auto W = [&](int i) { return (const bf16_t*)(lw + m->lay.off[i]); };
    T* kp = (T*)kv->k + l * kv_layer;
    T* vp = (T*)kv->v + l * kv_layer;
    if (l == 0)      // later layers: the previous layer's down projection normalised x already
      CALL(NOVA_KIND_MISC, s, nova::norm_rows<T>(x, S, H, W(0), nullptr, c.eps, 0, a, H, 1, 0, 0, s));
    {
      const GemmArgs p = with_split(GemmArgs{a, H, W(1), H, S, m->qkvw, H, nullptr, qkv, m->qkvw, nullptr, 0});
      CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_STORE, s)));
    }
    CALL(NOVA_KIND_MISC, s, nova::qkv_prefill<T>(qkv, S, 1, c.n_q, c.n_kv, D, c.rope_theta, 0, vt, skp, kp, vp, table,
                                                  c.block, s, att_cnt, n_cnt));
    {
      nova::AttnArgs p{qkv, m->qkvw, 0, qkv + qd, m->qkvw, 0, vt, skp, att, qd, 0, S, S, c.n_q, c.n_kv, 1, 1};
      // the split-K partials are free between the QKV and O projections: the attention's key
      // ranges keep theirs there
      p.part = split_ws, p.part_bytes = split_floats * sizeof(float), p.counters = att_cnt, p.cus = cus;
      CALL(NOVA_KIND_ATTN, s, nova::attention<T>(p, D, s));
    }
    if (int rc = resid_then_norm(with_split(GemmArgs{att, qd, W(2), qd, S, H, qd, nullptr, x, H, nullptr, 0}), W(3)))
      return rc;
    {
      GemmArgs p{a, H, W(4), H, S, 2 * m->ip, H, nullptr, hm, m->ip, nullptr, 0};
      CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_SWIGLU, s)));
    }
    {
      const GemmArgs p = with_split(GemmArgs{hm, m->ip, W(5), m->ip, S, H, m->ip, nullptr, x, H, nullptr, 0});
      if (l + 1 < c.layers) {   // with the next layer's input norm
        const bf16_t* next_gain = (const bf16_t*)((const char*)m->d.layers + (size_t)(l + 1) * m->lay.bytes + m->lay.off[0]);
        if (int rc = resid_then_norm(p, next_gain)) return rc;
      } else {                  // the last layer: the final norm reads the last row only
        CALL(NOVA_KIND_GEMM, s, (nova::gemm<T, T>(p, nova::EPI_RESID, s)));
      }
    }
  }
  const char* hw = (const char*)m->d.head;
  CALL(NOVA_KIND_MISC, s, nova::resid_rmsnorm<T>(nullptr, 0, x + (size_t)(S - 1) * H, 1, H,
                                                 (const bf16_t*)(hw + m->head.off[0]), c.eps, a, H, keys, s));
  {
    GemvArgs p{a, H, (const bf16_t*)(hw + m->head.off[1]), H, 1, c.vocab, H, logits_out, c.vocab, nullptr, keys};
    p.cus = cus;
    CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_ARGMAX, s)));
  }
  CALL(NOVA_KIND_MISC, s, nova::argmax_finish(keys, 1, next_id, s));
  return NOVA_OK;
}

template <typename T>
int llm_decode_t(const nova_llm* m, const int* ids, const int* pos, const int* tables, int max_blocks, int B, int max_ctx,
                 const nova_kv* kv, int* next_ids, float* logits_out, void* ws, hipStream_t s) {
  const nova_llm_config& c = m->d.cfg;
  const int H = c.hidden, D = c.head_dim, qd = c.n_q * D;
  const DecodeBufs<T> d = decode_bufs<T>(m, B, max_ctx, ws);
  const size_t kv_layer = (size_t)kv->num_blocks * c.n_kv * c.block * D;
  const bool f32 = sizeof(T) == 4;
  const int tiles = H / 64;
  const int cus = stream_cus(s);
  const int sp_qkv = nova::gemv_splits(m->qkvw, H, B, f32, cus);
  const char* hw = (const char*)m->d.head;
  auto layer_w = [&](int l, int i) {
    return (const bf16_t*)((const char*)m->d.layers + (size_t)l * m->lay.bytes + m->lay.off[i]);
  };
  const bf16_t* final_gain = (const bf16_t*)(hw + m->head.off[0]);
  auto attention_block = [&](int l) -> int {
    T* kp = (T*)kv->k + l * kv_layer;
    T* vp = (T*)kv->v + l * kv_layer;
    nova::DecAttnArgs p{sp_qkv > 1 ? d.part : d.qkv, sp_qkv, d.rope, kp, vp, tables, max_blocks, pos, d.att, d.apart,
                        B, c.n_q, c.n_kv, c.block, max_ctx};
    CALL(NOVA_KIND_DECODE_ATTN, s, nova::decode_attention<T>(p, D, s));
    return (int)NOVA_OK;
  };

  if (B <= 8) {
    // Small batches: each RMSNorm is folded into its neighbours.  The producer of the residual
    // (embedding, O and down projections) writes x times the norm's gain and per-tile sums of
    // squares of x, and the consumer projection (QKV, gate/up, LM head) scales each output by the
    // row's rsqrt.  (With larger batches the split-K tail of the producers outgrows a separate
    // norm kernel.)  The QKV split-K partials are summed by the decode attention, which also
    // applies the rotary embedding and appends the new k and v to the cache.
    auto ss = [&](int k) { return d.ss + (size_t)k * tiles * B; };
    CALL(NOVA_KIND_MISC, s, nova::decode_embed<T>(ids, B, (const bf16_t*)m->d.embed, H,
                                                  c.layers > 0 ? layer_w(0, 0) : final_gain, d.x, d.a, ss(0), tiles, d.keys,
                                                  d.counters, 2 * c.layers * tiles, pos, c.rope_theta, D, d.rope, s));
    for (int l = 0; l < c.layers; ++l) {
      auto W = [&](int i) { return layer_w(l, i); };
      {
        GemvArgs p{d.a, H, W(1), H, B, m->qkvw, H, sp_qkv > 1 ? nullptr : d.qkv, m->qkvw, d.part, nullptr};
        p.cus = cus;
        p.ss_in = ss(2 * l), p.ss_parts = tiles, p.eps = c.eps;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_STORE, s)));
      }
      if (const int rc = attention_block(l)) return rc;
      {
        GemvArgs p{d.att, qd, W(2), qd, B, H, qd, d.x, H, d.part, nullptr};
        p.cus = cus;
        p.ss_out = ss(2 * l + 1), p.counters = d.counters + (size_t)(2 * l) * tiles;
        p.gain_out = W(3), p.aout = d.a, p.ldao = H;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_RESID, s)));
      }
      {
        GemvArgs p{d.a, H, W(4), H, B, 2 * m->ip, H, d.hm, m->ip, d.part, nullptr};
        p.cus = cus;
        p.ss_in = ss(2 * l + 1), p.ss_parts = tiles, p.eps = c.eps;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, T>(p, nova::EPI_SWIGLU, s)));
      }
      {
        GemvArgs p{d.hm, m->ip, W(5), m->ip, B, H, m->ip, d.x, H, d.part, nullptr};
        p.cus = cus;
        p.ss_out = ss(2 * l + 2), p.counters = d.counters + (size_t)(2 * l + 1) * tiles;
        p.gain_out = l + 1 < c.layers ? layer_w(l + 1, 0) : final_gain, p.aout = d.a, p.ldao = H;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_RESID, s)));
      }
    }
    GemvArgs p{d.a, H, (const bf16_t*)(hw + m->head.off[1]), H, B, c.vocab, H, logits_out, c.vocab, d.part, d.keys};
    p.cus = cus;
    p.ss_in = ss(2 * c.layers), p.ss_parts = tiles, p.eps = c.eps;
    CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_ARGMAX, s)));
  } else {
    // Larger batches: a column-parallel fold kernel sums the O / down split-K partials into x,
    // writes x * gain and per-64-column sums of squares, and the consumer projections normalise
    // from those parts as above.
    const int sp_o = nova::gemv_splits(H, qd, B, f32, cus);
    const int sp_down = nova::gemv_splits(H, m->ip, B, f32, cus);
    auto ss = [&](int k) { return d.ss + (size_t)k * tiles * B; };
    CALL(NOVA_KIND_MISC, s, nova::decode_embed<T>(ids, B, (const bf16_t*)m->d.embed, H,
                                                  c.layers > 0 ? layer_w(0, 0) : final_gain, d.x, d.a, ss(0), tiles, d.keys,
                                                  nullptr, 0, pos, c.rope_theta, D, d.rope, s));
    for (int l = 0; l < c.layers; ++l) {
      auto W = [&](int i) { return layer_w(l, i); };
      {
        GemvArgs p{d.a, H, W(1), H, B, m->qkvw, H, sp_qkv > 1 ? nullptr : d.qkv, m->qkvw, d.part, nullptr};
        p.cus = cus;
        p.ss_in = ss(2 * l), p.ss_parts = tiles, p.eps = c.eps;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_STORE, s)));
      }
      if (const int rc = attention_block(l)) return rc;
      {
        GemvArgs p{d.att, qd, W(2), qd, B, H, qd, sp_o > 1 ? nullptr : d.x, H, d.part, nullptr};
        p.cus = cus;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_RESID, s)));
      }
      CALL(NOVA_KIND_MISC, s, nova::resid_fold<T>(sp_o > 1 ? d.part : nullptr, sp_o > 1 ? sp_o : 0, d.x, B, H, W(3), d.a, H,
                                                  ss(2 * l + 1), s));
      {
        GemvArgs p{d.a, H, W(4), H, B, 2 * m->ip, H, d.hm, m->ip, d.part, nullptr};
        p.cus = cus;
        p.ss_in = ss(2 * l + 1), p.ss_parts = tiles, p.eps = c.eps;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, T>(p, nova::EPI_SWIGLU, s)));
      }
      {
        GemvArgs p{d.hm, m->ip, W(5), m->ip, B, H, m->ip, sp_down > 1 ? nullptr : d.x, H, d.part, nullptr};
        p.cus = cus;
        CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_RESID, s)));
      }
      CALL(NOVA_KIND_MISC, s, nova::resid_fold<T>(sp_down > 1 ? d.part : nullptr, sp_down > 1 ? sp_down : 0, d.x, B, H,
                                                  l + 1 < c.layers ? layer_w(l + 1, 0) : final_gain, d.a, H,
                                                  ss(2 * l + 2), s));
    }
    GemvArgs p{d.a, H, (const bf16_t*)(hw + m->head.off[1]), H, B, c.vocab, H, logits_out, c.vocab, d.part, d.keys};
    p.cus = cus;
    p.ss_in = ss(2 * c.layers), p.ss_parts = tiles, p.eps = c.eps;
    CALL(NOVA_KIND_GEMV, s, (nova::gemv<T, float>(p, nova::EPI_ARGMAX, s)));
  }
  CALL(NOVA_KIND_MISC, s, nova::argmax_finish(d.keys, B, next_ids, s));
  return NOVA_OK;
}
}  // namespace

extern "C" int nova_llm_prefill(const nova_llm* m, const void* vis, int n_vis, const int32_t* ids, int n_text,
                                const int32_t* table, const nova_kv* kv, int32_t* next_id, float* logits, void* ws,
                                size_t ws_bytes, nova_stream_t stream) {
  if (!m || !kv) return fail(NOVA_EINVAL, "null model or kv");
  if (n_vis < 0 || n_text < 0 || n_vis + n_text <= 0) return fail(NOVA_EINVAL, "empty prompt");
  if ((n_vis > 0 && (!vis || !aligned(vis))) || (n_text > 0 && !ids) || !table || !next_id || !ws || !aligned(ws))
    return fail(NOVA_EINVAL, "null or misaligned pointer");
  if (!kv->k || !kv->v || kv->num_blocks <= 0) return fail(NOVA_EINVAL, "invalid kv pool");
  const int S = n_vis + n_text;
  if ((S + m->d.cfg.block - 1) / m->d.cfg.block > kv->num_blocks) return fail(NOVA_ENOKV, "prompt needs more blocks than the pool holds");
  const size_t need = nova_llm_prefill_workspace_bytes(m, S);
  if (ws_bytes < need) return fail(NOVA_ENOSPACE, "workspace %zu < required %zu bytes", ws_bytes, need);
  hipStream_t s = (hipStream_t)stream;
  return m->d.cfg.act == NOVA_ACT_F32
             ? llm_prefill_t<float>(m, (const float*)vis, n_vis, ids, n_text, table, kv, next_id, logits, ws, s)
             : llm_prefill_t<bf16_t>(m, (const bf16_t*)vis, n_vis, ids, n_text, table, kv, next_id, logits, ws, s);
}

namespace {
// Argument checks shared by the two decode entry points (everything but the workspace).
int check_decode_args(const nova_llm* m, const int32_t* ids, const int32_t* pos, const int32_t* tables, int max_blocks,
                      int batch, int max_ctx, const nova_kv* kv, const int32_t* next_ids) {
  if (!m || !kv) return fail(NOVA_EINVAL, "null model or kv");
  if (batch <= 0 || batch > 32) return fail(NOVA_EINVAL, "batch %d outside 1..32", batch);
  if (!ids || !pos || !tables || !next_ids) return fail(NOVA_EINVAL, "null pointer");
  if (max_ctx <= 0 || max_blocks <= 0) return fail(NOVA_EINVAL, "max_ctx and max_blocks must be positive");
  if ((max_ctx + m->d.cfg.block - 1) / m->d.cfg.block > max_blocks) return fail(NOVA_ENOKV, "max_ctx exceeds the block table width");
  if (!kv->k || !kv->v || kv->num_blocks <= 0) return fail(NOVA_EINVAL, "invalid kv pool");
  return NOVA_OK;
}

int decode_dispatch(const nova_llm* m, const int32_t* ids, const int32_t* pos, const int32_t* tables, int max_blocks,
                    int batch, int max_ctx, const nova_kv* kv, int32_t* next_ids, float* logits, void* ws,
                    hipStream_t s) {
  return m->d.cfg.act == NOVA_ACT_F32
             ? llm_decode_t<float>(m, ids, pos, tables, max_blocks, batch, max_ctx, kv, next_ids, logits, ws, s)
             : llm_decode_t<bf16_t>(m, ids, pos, tables, max_blocks, batch, max_ctx, kv, next_ids, logits, ws, s);
}
}  // namespace

extern "C" int nova_llm_decode(const nova_llm* m, const int32_t* ids, const int32_t* pos, const int32_t* tables,
                               int max_blocks, int batch, int max_ctx, const nova_kv* kv, int32_t* next_ids,
                               float* logits, void* ws, size_t ws_bytes, nova_stream_t stream) {
  if (int rc = check_decode_args(m, ids, pos, tables, max_blocks, batch, max_ctx, kv, next_ids)) return rc;
  if (!ws || !aligned(ws)) return fail(NOVA_EINVAL, "null or misaligned workspace");
  const size_t need = nova_llm_decode_workspace_bytes(m, batch, max_ctx);
  if (ws_bytes < need) return fail(NOVA_ENOSPACE, "workspace %zu < required %zu bytes", ws_bytes, need);
  return decode_dispatch(m, ids, pos, tables, max_blocks, batch, max_ctx, kv, next_ids, logits, ws, (hipStream_t)stream);
}

// ------------------------------------------------------------------ allocation-free decode
// The decode workspace of nova_llm_decode_noalloc: one static device array, which every GPU the
// library runs on holds at its own address until the process ends.  Host code never passes the
// array's name to a kernel or a copy (on the host it only stands in for the symbol); it uses the
// device address that hipGetSymbolAddress returns, once per device, with that device current.
static __device__ __align__(256) unsigned char scratch[NOVA_DECODE_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (resolved on first use per device).
int scratch_for_current_device(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(NOVA_EUNSUPPORTED, "device %d beyond the scratch table", dev);
  std::lock_guard<std::mutex> lk(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return fail(NOVA_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    scratch_ptr[dev] = ptr;
  }
  *out = scratch_ptr[dev];
  return NOVA_OK;
}
}  // namespace

extern "C" int nova_llm_decode_noalloc(const nova_llm* m, const int32_t* ids, const int32_t* pos,
                                       const int32_t* tables, int max_blocks, int batch, int max_ctx,
                                       const nova_kv* kv, int32_t* next_ids, float* logits, nova_stream_t stream) {
  if (int rc = check_decode_args(m, ids, pos, tables, max_blocks, batch, max_ctx, kv, next_ids)) return rc;
  const size_t need = nova_llm_decode_workspace_bytes(m, batch, max_ctx);
  if (need > (size_t)NOVA_DECODE_SCRATCH_BYTES)
    return fail(NOVA_ENOSPACE, "decode step needs %zu bytes of workspace, above the %zu-byte static scratch "
                               "(use nova_llm_decode with a caller workspace)", need, (size_t)NOVA_DECODE_SCRATCH_BYTES);
  void* ws = nullptr;
  if (int rc = scratch_for_current_device(&ws)) return rc;
  // the step clears what must start at zero (argmax keys, arrival counters) in its first kernel
  return decode_dispatch(m, ids, pos, tables, max_blocks, batch, max_ctx, kv, next_ids, logits, ws, (hipStream_t)stream);
}

// ------------------------------------------------------------------ linear co-run study
extern "C" int nova_linear(int variant, const void* x, int M, int K, const void* w, int N, float* out,
                           nova_stream_t stream) {
  if (!x || !w || !out || !aligned(x) || !aligned(w) || !aligned(out))
    return fail(NOVA_EINVAL, "x, w and out must be non-null and 256-byte aligned");
  if (M <= 0 || N <= 0 || K <= 0) return fail(NOVA_EINVAL, "non-positive size");
  hipStream_t s = (hipStream_t)stream;
  const bf16_t* xb = (const bf16_t*)x;
  const bf16_t* wb = (const bf16_t*)w;
  switch (variant) {
    case NOVA_LINEAR_TILED:
    case NOVA_LINEAR_TILED_SMALL: {
      if (K % 64 || N % 128) return fail(NOVA_EUNSUPPORTED, "tiled linear needs K %% 64 == 0 and N %% 128 == 0");
      GemmArgs p{xb, K, wb, K, M, N, K, nullptr, out, N, nullptr, 0};
      p.small_tiles = variant == NOVA_LINEAR_TILED_SMALL;
      CALL(NOVA_KIND_GEMM, s, (nova::gemm<bf16_t, bf16_t>(p, nova::EPI_RESID, s)));
      return NOVA_OK;
    }
    case NOVA_LINEAR_THIN: {
      const int cus = stream_cus(s);
      if (M > 32 || K % 256 || N % 64) return fail(NOVA_EUNSUPPORTED, "thin linear needs M <= 32, K %% 256 == 0, N %% 64 == 0");
      if (nova::gemv_splits(N, K, M, false, cus) != 1)
        return fail(NOVA_EUNSUPPORTED, "thin linear of %d rows would split K on %d CUs (no workspace here)", N, cus);
      GemvArgs p{xb, K, wb, K, M, N, K, out, N, nullptr, nullptr};
      p.cus = cus;
      CALL(NOVA_KIND_GEMV, s, (nova::gemv<bf16_t, float>(p, nova::EPI_RESID, s)));
      return NOVA_OK;
    }
    case NOVA_LINEAR_THIN_VALU:
      if (M > 4 || K % 512) return fail(NOVA_EUNSUPPORTED, "vector-ALU linear needs M <= 4 and K %% 512 == 0");
      CALL(NOVA_KIND_GEMV, s, nova::gemv_valu(xb, K, wb, K, M, N, K, out, N, s));
      return NOVA_OK;
  }
  return fail(NOVA_EINVAL, "unknown linear variant %d", variant);
}

// ------------------------------------------------------------------ CU partitions
extern "C" int nova_make_cu_mask(int n_cus, int first_slot, uint32_t* mask) {
  if (!mask) return fail(NOVA_EINVAL, "null mask");
  if (n_cus <= 0 || n_cus % 8 || n_cus > 256) return fail(NOVA_EINVAL, "n_cus %d must be a positive multiple of 8 <= 256", n_cus);
  const int per_xcd = n_cus / 8;
  if (first_slot < 0 || first_slot + per_xcd > 32) return fail(NOVA_EINVAL, "slots %d..%d exceed 32 per XCD", first_slot, first_slot + per_xcd - 1);
  for (int w = 0; w < 8; ++w) mask[w] = 0u;
  // per-XCD slot s: engine s % 4, CU s / 4 of that engine -> bit 32*(s/4) + 8*(s%4) + xcd
  for (int s = first_slot; s < first_slot + per_xcd; ++s)
    for (int xcd = 0; xcd < 8; ++xcd) {
      const int bit = 32 * (s / 4) + 8 * (s % 4) + xcd;
      mask[bit / 32] |= 1u << (bit % 32);
    }
  return NOVA_OK;
}

namespace {
// Each CU-masked stream holds a hardware queue of its own, and past about a dozen of them in one
// process every queue's work slows down, idle ones included (measured: the whole-GPU 8-image encode
// on another stream 89 ms with 12 masked streams alive, 156 ms with 24, 705 ms with 140).  The pool
// therefore keeps at most this many; before it grows past that, the least recently used streams
// that no stage holds are drained and destroyed (a caller keeps a stage's stream until its next
// partition call for that stage, which is never evicted).
constexpr size_t kMaxMaskStreams = 8;

void make_room_for_mask_streams(const std::vector<uint32_t>& keep) {
  std::vector<uint32_t> comp(8);
  for (int w = 0; w < 8; ++w) comp[w] = ~keep[w];
  while (g.mask_streams.size() + 2 > kMaxMaskStreams) {
    const std::vector<uint32_t>* victim = nullptr;
    uint64_t oldest = ~0ull;
    for (auto& kv : g.mask_streams) {
      bool held = kv.first == keep || kv.first == comp;
      for (int st = 0; st < 3 && !held; ++st) held = g.stage_stream[st] == kv.second;
      const uint64_t u = g.mask_used[kv.first];
      if (!held && u < oldest) { oldest = u; victim = &kv.first; }
    }
    if (!victim) return;                  // every pooled stream is held: grow past the cap
    const std::vector<uint32_t> v = *victim;
    hipStream_t s = g.mask_streams[v];
    hipStreamSynchronize(s);
    hipStreamDestroy(s);
    g.mask_streams.erase(v);
    g.mask_used.erase(v);
  }
}
}  // namespace

extern "C" int nova_set_stage_partition(int stage, const uint32_t* cu_mask, int mask_words, nova_stream_t* out_stream) {
  if (stage < 0 || stage > 2) return fail(NOVA_EINVAL, "stage %d out of range", stage);
  if (!cu_mask || !out_stream || mask_words <= 0 || mask_words > 8) return fail(NOVA_EINVAL, "mask needs 1..8 words");
  if (g.device < 0) return fail(NOVA_EINVAL, "nova_init not called");
  std::vector<uint32_t> m(8, 0u);
  for (int i = 0; i < mask_words; ++i) m[i] = cu_mask[i];
  // every XCD (bit i -> XCD i % 8) must keep at least one CU, or its share of a kernel's
  // workgroups could never be scheduled
  for (int xcd = 0; xcd < 8; ++xcd) {
    bool any = false;
    for (int bit = xcd; bit < 256 && !any; bit += 8) any = (m[bit / 32] >> (bit % 32)) & 1u;
    if (!any) return fail(NOVA_EINVAL, "mask leaves XCD %d without compute units", xcd);
  }
  std::lock_guard<std::mutex> lk(g.mu);
  hipStream_t ns;
  // the whole-GPU mask is the one two stages may hold at once (a stage keeps a pass's stream
  // until the pass ends): it gets one stream per stage, created together
  bool full = true;
  for (int w = 0; w < 8; ++w) full = full && m[w] == 0xFFFFFFFFu;
  if (full) {
    if (!g.full_streams[stage]) {
      for (int st = 0; st < 3; ++st) {
        if (g.full_streams[st]) continue;
        hipError_t e = hipExtStreamCreateWithCUMask(&g.full_streams[st], 8, m.data());
        if (e != hipSuccess) return fail(NOVA_EHIP, "hipExtStreamCreateWithCUMask: %s", hipGetErrorString(e));
      }
    }
    ns = g.full_streams[stage];
  } else if (g.mask_streams.find(m) == g.mask_streams.end()) {
    make_room_for_mask_streams(m);
    hipError_t e = hipExtStreamCreateWithCUMask(&ns, 8, m.data());
    if (e != hipSuccess) return fail(NOVA_EHIP, "hipExtStreamCreateWithCUMask: %s", hipGetErrorString(e));
    g.mask_streams[m] = ns;
    // Co-running stages hold complementary masks.  Hardware queues are dealt to the command
    // processor's dispatch pipes as they are created, and two queues on one pipe take turns:
    // a kernel with more workgroups than fit keeps its pipe busy until its last workgroup is
    // placed, stalling the other queue.  Creating the complement's queue right after this one
    // puts the pair on different pipes.
    std::vector<uint32_t> c(8);
    bool every_xcd = true;
    for (int w = 0; w < 8; ++w) c[w] = ~m[w];
    for (int xcd = 0; xcd < 8 && every_xcd; ++xcd) {
      bool any = false;
      for (int bit = xcd; bit < 256 && !any; bit += 8) any = (c[bit / 32] >> (bit % 32)) & 1u;
      every_xcd = any;
    }
    if (every_xcd && g.mask_streams.find(c) == g.mask_streams.end()) {
      hipStream_t cs;
      e = hipExtStreamCreateWithCUMask(&cs, 8, c.data());
      if (e != hipSuccess) return fail(NOVA_EHIP, "hipExtStreamCreateWithCUMask: %s", hipGetErrorString(e));
      g.mask_streams[c] = cs;
      g.mask_used[c] = ++g.uses;
    }
  } else {
    ns = g.mask_streams[m];
  }
  if (!full) g.mask_used[m] = ++g.uses;
  hipStream_t old = g.stage_stream[stage];
  if (old && old != ns) {
    if (!g.stage_switch[stage]) HIP_TRY(hipEventCreateWithFlags(&g.stage_switch[stage], hipEventDisableTiming));
    HIP_TRY(hipEventRecord(g.stage_switch[stage], old));
    HIP_TRY(hipStreamWaitEvent(ns, g.stage_switch[stage], 0));
  }
  g.stage_stream[stage] = ns;
  *out_stream = (nova_stream_t)ns;
  return NOVA_OK;
}

extern "C" int nova_cu_probe(nova_stream_t stream, uint32_t* out, int n) {
  if (!out || n <= 0) return fail(NOVA_EINVAL, "cu_probe needs an output array and n > 0");
  HIP_TRY(nova::cu_probe((hipStream_t)stream, out, n));
  return NOVA_OK;
}

// ------------------------------------------------------------------ timing
extern "C" int nova_timing_enable(int on) {
  g.timing = on != 0;
  return NOVA_OK;
}

extern "C" int nova_timing_read(int kind, double* total_ms, int* launches) {
  if (kind < 0 || kind > NOVA_KIND_MISC || !total_ms || !launches) return fail(NOVA_EINVAL, "bad timing query");
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
  {
    std::lock_guard<std::mutex> lk(g.mu);
    ev.swap(g.ev_used[kind]);
  }
  double tot = 0.0;
  int rc = NOVA_OK;
  for (auto& pr : ev) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(pr.second);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, pr.first, pr.second);
    if (e != hipSuccess && rc == NOVA_OK) rc = fail(NOVA_EHIP, "event timing: %s", hipGetErrorString(e));
    tot += ms;
  }
  {
    std::lock_guard<std::mutex> lk(g.mu);
    for (auto& pr : ev) { g.ev_free.push_back(pr.first); g.ev_free.push_back(pr.second); }
  }
  *total_ms = tot;
  *launches = (int)ev.size();
  return rc;
}
