// Memory-bound glue kernels of the three stages: LayerNorm/RMSNorm (with the 2x2 patch-merge
// scatter fused into the LayerNorm store), patchify, QKV split with rotary embedding, transposed
// V and paged-cache writes, embedding gather and greedy argmax.  All use 16-byte coalesced
// accesses along the hidden dimension; statistics are accumulated in fp32.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace nova {

// ------------------------------------------------------------------ norms (one wave per row)
// LayerNorm (ln = 1, with shift) or RMSNorm (ln = 0) of fp32 rows of width H <= 4096: the row is
// read once into registers (lane l holds float4 l, l + 64, ...), mean and variance come from the
// registers (two passes over them, so the variance is well conditioned), and each lane writes 4
// outputs at a time.  merge > 1 scatters row (image, py, px) of a gh x gw patch grid to the
// merged token it belongs to, at column block (py % merge) * merge + px % merge.
constexpr int NORM_MAXV = 16;     // float4 per lane: H <= 64 * 4 * 16
// NV: float4 per lane held in registers (the row width rounded up to 256 columns), as few as the
// row needs so that more rows are in flight per CU
// RES: before the statistics, the row is updated in place with a residual branch that arrives as
// `slices` fp32 K-slice partials (part + k * pstride, k = 0 .. slices-1, summed in slice order, as
// split_reduce_kernel does): x += ((p_0 + p_1) + ...).  This folds the reduction pass of a K-split
// residual projection into the norm that reads its output next.
template <typename T, int NV, bool RES>
__global__ void __launch_bounds__(256) norm_kernel(float* __restrict__ x, int M, int H, const bf16_t* __restrict__ g,
                                                   const bf16_t* __restrict__ bb, float eps, int ln, T* __restrict__ out,
                                                   int ldo, int merge, int gh, int gw, const float* __restrict__ part,
                                                   int slices, size_t pstride) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  float4* xr = reinterpret_cast<float4*>(x + (size_t)row * H);
  const int n4 = H / 4;
  // every load of a phase is issued before any of its values is used: the gain (and, without a
  // residual branch, the shift), x and the first partial slice together, then each further
  // slice; a load issued after a store of x would wait for the stores before it (one round trip
  // to memory per chunk)
  uint2 gg[NV], bs[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = j * 64 + lane;
    gg[j] = i < n4 ? *reinterpret_cast<const uint2*>(g + 4 * i) : make_uint2(0u, 0u);
    if constexpr (!RES) bs[j] = ln && i < n4 ? *reinterpret_cast<const uint2*>(bb + 4 * i) : make_uint2(0u, 0u);
  }
  float4 v[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = j * 64 + lane;
    v[j] = i < n4 ? xr[i] : float4{0.f, 0.f, 0.f, 0.f};
  }
  if constexpr (RES) {
    const float4* pr = reinterpret_cast<const float4*>(part + (size_t)row * H);
    float4 d[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int i = j * 64 + lane;
      d[j] = i < n4 ? pr[i] : float4{0.f, 0.f, 0.f, 0.f};
    }
    for (int k = 1; k < slices; ++k) {
      float4 e[NV];
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int i = j * 64 + lane;
        e[j] = i < n4 ? pr[k * (pstride / 4) + i] : float4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int j = 0; j < NV; ++j) d[j] = float4{d[j].x + e[j].x, d[j].y + e[j].y, d[j].z + e[j].z, d[j].w + e[j].w};
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int i = j * 64 + lane;
      v[j] = float4{v[j].x + d[j].x, v[j].y + d[j].y, v[j].z + d[j].z, v[j].w + d[j].w};
      if (i < n4) xr[i] = v[j];
    }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) s += v[j].x + v[j].y + v[j].z + v[j].w;
  const float mean = ln ? wave_sum(s) / H : 0.f;
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    if (j * 64 + lane < n4) {
      const float a = v[j].x - mean, b = v[j].y - mean, c = v[j].z - mean, d = v[j].w - mean;
      ss += a * a + b * b + c * c + d * d;
    }
  }
  const float rstd = rsqrtf(wave_sum(ss) / H + eps);
  size_t orow = row, ocol = 0;
  if (merge > 1) {
    const int per_img = gh * gw;
    const int img = row / per_img, r = row % per_img, py = r / gw, px = r % gw;
    orow = (size_t)img * (per_img / (merge * merge)) + (py / merge) * (gw / merge) + px / merge;
    ocol = (size_t)((py % merge) * merge + px % merge) * H;
  }
  T* o = out + orow * ldo + ocol;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = j * 64 + lane;
    if (i >= n4) continue;
    float y[4] = {(v[j].x - mean) * rstd * bf2f((bf16_t)(gg[j].x & 0xffff)), (v[j].y - mean) * rstd * bf2f((bf16_t)(gg[j].x >> 16)),
                  (v[j].z - mean) * rstd * bf2f((bf16_t)(gg[j].y & 0xffff)), (v[j].w - mean) * rstd * bf2f((bf16_t)(gg[j].y >> 16))};
    if (ln) {
      const uint2 b2 = RES ? *reinterpret_cast<const uint2*>(bb + 4 * i) : bs[j];
      y[0] += bf2f((bf16_t)(b2.x & 0xffff)); y[1] += bf2f((bf16_t)(b2.x >> 16));
      y[2] += bf2f((bf16_t)(b2.y & 0xffff)); y[3] += bf2f((bf16_t)(b2.y >> 16));
    }
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<float4*>(o + 4 * i) = float4{y[0], y[1], y[2], y[3]};
    } else {
      *reinterpret_cast<uint2*>(o + 4 * i) = make_uint2(pack2(y[0], y[1]), pack2(y[2], y[3]));
    }
  }
}

template <typename T, bool RES>
static hipError_t norm_launch(float* x, int M, int H, const bf16_t* g, const bf16_t* b, float eps, int ln, T* out, int ldo,
                              int merge, int gh, int gw, const float* part, int slices, size_t pstride, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (H % 4 || H > 4 * 64 * NORM_MAXV || ldo % 4) return hipErrorInvalidValue;
  const dim3 grid((M + 3) / 4);
  const int nv = (H + 255) / 256;
#define NORM_LAUNCH(NVV)                                                                                             \
  hipLaunchKernelGGL((norm_kernel<T, NVV, RES>), grid, dim3(256), 0, s, x, M, H, g, b, eps, ln, out, ldo, merge, gh, gw, \
                     part, slices, pstride)
  if (nv <= 1) NORM_LAUNCH(1);
  else if (nv <= 2) NORM_LAUNCH(2);
  else if (nv <= 4) NORM_LAUNCH(4);
  else if (nv <= 5) NORM_LAUNCH(5);
  else if (nv <= 8) NORM_LAUNCH(8);
  else if (nv <= 14) NORM_LAUNCH(14);
  else NORM_LAUNCH(NORM_MAXV);
#undef NORM_LAUNCH
  return hipGetLastError();
}

template <typename T>
hipError_t norm_rows(const float* x, int M, int H, const bf16_t* g, const bf16_t* b, float eps, int ln, T* out,
                     int ldo, int merge, int gh, int gw, hipStream_t s) {
  // the plain norm never writes x
  return norm_launch<T, false>(const_cast<float*>(x), M, H, g, b, eps, ln, out, ldo, merge, gh, gw, nullptr, 0, 0, s);
}

template <typename T>
hipError_t split_norm_rows(const float* part, int slices, size_t pstride, float* x, int M, int H, const bf16_t* g,
                           const bf16_t* b, float eps, int ln, T* out, int ldo, hipStream_t s) {
  if (part == nullptr || slices < 1 || pstride < (size_t)M * H || pstride % 4) return hipErrorInvalidValue;
  return norm_launch<T, true>(x, M, H, g, b, eps, ln, out, ldo, 1, 0, 0, part, slices, pstride, s);
}

// ------------------------------------------------------------------ patchify
template <typename T>
__global__ void patchify_kernel(const bf16_t* __restrict__ img, int B, int H, int W, int p, int kpad, T* __restrict__ out) {
  const int gw = W / p, gh = H / p;
  const long total = (long)B * gh * gw * kpad;
  for (long idx = (long)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += (long)gridDim.x * blockDim.x) {
    const int col = (int)(idx % kpad);
    const long prow = idx / kpad;
    float v = 0.f;
    if (col < 3 * p * p) {
      const int c = col % 3, px = (col / 3) % p, py = col / (3 * p);
      const int img_i = (int)(prow / (gh * gw)), r = (int)(prow % (gh * gw));
      const int y = (r / gw) * p + py, x = (r % gw) * p + px;
      v = bf2f(img[(((size_t)img_i * H + y) * W + x) * 3 + c]);
    }
    out[idx] = from_f<T>(v);
  }
}

template <typename T>
hipError_t patchify(const bf16_t* img, int B, int H, int W, int p, int kpad, T* out, hipStream_t s) {
  const long total = (long)B * (H / p) * (W / p) * kpad;
  if (total <= 0) return hipSuccess;
  const int grid = (int)std::min<long>((total + 255) / 256, 65536);
  hipLaunchKernelGGL((patchify_kernel<T>), dim3(grid), dim3(256), 0, s, img, B, H, W, p, kpad, out);
  return hipGetLastError();
}

// ------------------------------------------------------------------ projected rows -> attention inputs
// One pass over the packed QKV rows of a prefill (or a bidirectional encode): workgroup (64-token
// tile, head, batch) of a grid over every q, k and v head.
//  * q and k heads (rope_theta > 0): rotary embedding in place, half-split pairing (c, c + D/2)
//    by angle pos * theta^(-2c/D); a thread takes one 16-byte piece of each half (8 bf16 or 4 fp32
//    pairs); the inverse frequencies are computed once per workgroup and each angle is formed and
//    reduced in double before the fp32 sine/cosine, as in the decode step's table.  A k head also
//    appends its rotated rows to the paged cache K [blk][kvh][slot][D] (16-byte pieces).
//  * v heads: V^T [b][kv head][D][sk_pad] for the attention kernel (keys past S zero) and the
//    paged V [blk][kvh][D][slot], through an LDS tile: 16-byte reads of each token's D values,
//    16-byte writes of 16 / sizeof(T) consecutive keys of each V^T row.
template <typename T>
__global__ void __launch_bounds__(256) qkv_prefill_kernel(T* __restrict__ qkv, int S, int n_q, int n_kv, int D, float theta,
                                                          int pos0, T* __restrict__ vt, int sk_pad, T* __restrict__ kpool,
                                                          T* __restrict__ vpool, const int* __restrict__ table, int block,
                                                          int h0, unsigned* __restrict__ zero, int nzero) {
  constexpr int EPC = 16 / sizeof(T);      // elements per 16-byte piece
  if (zero != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0)
    for (int i = threadIdx.x; i < nzero; i += 256) zero[i] = 0u;
  constexpr int TP = 128 + EPC;            // tile pitch (elements), D <= 128
  __shared__ __align__(16) T tile[64 * TP];
  __shared__ double inv_s[64];             // D / 2 <= 64
  const int t0 = blockIdx.x * 64, hh = h0 + blockIdx.y, b = blockIdx.z;
  const int ld = (n_q + 2 * n_kv) * D;
  T* rows = qkv + (size_t)b * S * ld + (size_t)hh * D;
  if (hh < n_q + n_kv) {
    const bool khead = hh >= n_q;
    if (theta <= 0.f) {
      if (!khead || table == nullptr) return;
      // no rotation: the k rows go to the cache as they are
      for (int i = threadIdx.x; i < 64 * (D / EPC); i += 256) {
        const int t = i / (D / EPC), c = (i % (D / EPC)) * EPC, tok = t0 + t;
        if (tok >= S) continue;
        const int phys = table[tok / block], slot = tok % block;
        *reinterpret_cast<u32x4*>(kpool + (((size_t)phys * n_kv + (hh - n_q)) * block + slot) * D + c) =
            *reinterpret_cast<const u32x4*>(rows + (size_t)tok * ld + c);
      }
      return;
    }
    const int half = D / 2, pieces = half / EPC;
    for (int c = threadIdx.x; c < half; c += 256) inv_s[c] = exp2(-(2.0 * c / D) * log2((double)theta));
    __syncthreads();
    for (int i = threadIdx.x; i < 64 * pieces; i += 256) {
      const int t = i / pieces, pc = i % pieces, tok = t0 + t;
      if (tok >= S) continue;
      T* e1 = rows + (size_t)tok * ld + pc * EPC;
      T* e2 = e1 + half;
      T a[EPC], bv[EPC];
      *reinterpret_cast<u32x4*>(a) = *reinterpret_cast<const u32x4*>(e1);
      *reinterpret_cast<u32x4*>(bv) = *reinterpret_cast<const u32x4*>(e2);
      const double pos = (double)(pos0 + tok);
#pragma unroll
      for (int v = 0; v < EPC; ++v) {
        double ang = pos * inv_s[pc * EPC + v];
        ang -= 6.283185307179586 * floor(ang * 0.15915494309189535);
        float sn, cs;
        sincosf((float)ang, &sn, &cs);
        const float x1 = to_f<T>(a[v]), x2 = to_f<T>(bv[v]);
        a[v] = from_f<T>(x1 * cs - x2 * sn);
        bv[v] = from_f<T>(x2 * cs + x1 * sn);
      }
      *reinterpret_cast<u32x4*>(e1) = *reinterpret_cast<const u32x4*>(a);
      *reinterpret_cast<u32x4*>(e2) = *reinterpret_cast<const u32x4*>(bv);
      if (khead && table != nullptr) {
        T* kd = kpool + (((size_t)table[tok / block] * n_kv + (hh - n_q)) * block + tok % block) * D + pc * EPC;
        *reinterpret_cast<u32x4*>(kd) = *reinterpret_cast<const u32x4*>(a);
        *reinterpret_cast<u32x4*>(kd + half) = *reinterpret_cast<const u32x4*>(bv);
      }
    }
    return;
  }
  const int kvh = hh - n_q - n_kv;
  const int cpr = D / EPC;
  for (int c = threadIdx.x; c < 64 * cpr; c += 256) {
    const int t = c / cpr, d0 = (c % cpr) * EPC;
    u32x4 val = {0u, 0u, 0u, 0u};
    if (t0 + t < S) val = *reinterpret_cast<const u32x4*>(rows + (size_t)(t0 + t) * ld + d0);
    *reinterpret_cast<u32x4*>(tile + t * TP + d0) = val;
  }
  __syncthreads();
  T* vdst = vt + ((size_t)b * n_kv + kvh) * D * (size_t)sk_pad;
  constexpr int TCN = 64 / EPC;            // key pieces per V^T row of this tile
  for (int c = threadIdx.x; c < D * TCN; c += 256) {
    const int d = c / TCN, tc = (c % TCN) * EPC;
    T vals[EPC];
#pragma unroll
    for (int j = 0; j < EPC; ++j) vals[j] = tile[(tc + j) * TP + d];
    *reinterpret_cast<u32x4*>(vdst + (size_t)d * sk_pad + t0 + tc) = *reinterpret_cast<const u32x4*>(vals);
    // the same EPC keys of row d also form one piece of the paged V block ([d][slot] layout);
    // EPC divides the block, so the piece never straddles two blocks
    if (table != nullptr && t0 + tc < S) {
      const int tok = t0 + tc, phys = table[tok / block], slot = tok % block;
      if (tok + EPC <= S) {
        *reinterpret_cast<u32x4*>(vpool + (((size_t)phys * n_kv + kvh) * D + d) * block + slot) =
            *reinterpret_cast<const u32x4*>(vals);
      } else {
        for (int j = 0; j < S - tok; ++j) vpool[(((size_t)phys * n_kv + kvh) * D + d) * block + slot + j] = vals[j];
      }
    }
  }
}

template <typename T>
hipError_t qkv_prefill(T* qkv, int S, int batch, int n_q, int n_kv, int D, float rope_theta, int pos0, T* vt,
                       int sk_pad, T* kpool, T* vpool, const int* table, int block, hipStream_t s, unsigned* zero,
                       int nzero) {
  if (S <= 0) return hipSuccess;
  if (D > 128 || D % 16 || sk_pad < S || sk_pad % 64) return hipErrorInvalidValue;
  if (table != nullptr && block % (16 / (int)sizeof(T))) return hipErrorInvalidValue;
  // with no rotation and no cache, only the v heads have work
  const int h0 = rope_theta > 0.f || table != nullptr ? 0 : n_q + n_kv;
  dim3 grid(sk_pad / 64, n_q + 2 * n_kv - h0, batch);
  hipLaunchKernelGGL((qkv_prefill_kernel<T>), grid, dim3(256), 0, s, qkv, S, n_q, n_kv, D, rope_theta, pos0, vt, sk_pad,
                     kpool, vpool, table, block, h0, zero, nzero);
  return hipGetLastError();
}

// ------------------------------------------------------------------ decode residual + RMSNorm
// One 1024-thread workgroup per row: fold the split-K partials of the previous projection into
// the fp32 residual stream, then normalise the row for the next projection.
template <typename T>
__global__ void __launch_bounds__(1024) resid_rmsnorm_kernel(const float* __restrict__ partial, int splits,
                                                             float* __restrict__ x, int H, const bf16_t* __restrict__ g,
                                                             float eps, T* __restrict__ a, int lda,
                                                             unsigned long long* __restrict__ keys) {
  __shared__ float red[16];
  const int b = blockIdx.x, B = gridDim.x;
  if (keys != nullptr && threadIdx.x == 0) keys[b] = 0ull;
  float* xr = x + (size_t)b * H;
  float ss = 0.f;
  for (int c = threadIdx.x; c < H; c += blockDim.x) {
    float v = xr[c];
    if (splits > 0) {
      float acc = 0.f;
#pragma unroll 8
      for (int sp = 0; sp < splits; ++sp) acc += partial[((size_t)sp * B + b) * H + c];
      v += acc;
      xr[c] = v;
    }
    ss += v * v;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) tot += red[w];
  const float rstd = rsqrtf(tot / H + eps);
  for (int c = threadIdx.x; c < H; c += blockDim.x) a[(size_t)b * lda + c] = from_f<T>(xr[c] * rstd * bf2f(g[c]));
}

template <typename T>
hipError_t resid_rmsnorm(const float* partial, int splits, float* x, int B, int H, const bf16_t* g, float eps, T* a,
                         int lda, unsigned long long* keys, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL((resid_rmsnorm_kernel<T>), dim3(B), dim3(1024), 0, s, partial, splits, x, H, g, eps, a, lda, keys);
  return hipGetLastError();
}

// Decode residual fold for larger batches, spread over the whole GPU: workgroup (t, r) takes
// columns 64t .. 64t+63 of rows 8r .. 8r+7, one 32-lane half-wave per row and two columns per
// lane.  x[b] += sum_s partial[s][b] (if splits > 0), a[b] = x[b] * g, and the tile's sum of
// squares of x[b] goes to ss_out[t * B + b]; the normalising consumer sums the H / 64 tile parts
// and scales its outputs by the row's rsqrt.
template <typename T>
__global__ void __launch_bounds__(256) resid_fold_kernel(const float* __restrict__ partial, int splits,
                                                         float* __restrict__ x, int B, int H,
                                                         const bf16_t* __restrict__ g, T* __restrict__ a, int lda,
                                                         float* __restrict__ ss_out) {
  const int t = threadIdx.x, b = blockIdx.y * 8 + (t >> 5);
  const int c = blockIdx.x * 64 + (t & 31) * 2;
  float sq = 0.f;
  if (b < B) {
    // the gain pair is loaded with x and the partials (the compiler would otherwise issue it
    // after the store of x, a second round trip to memory)
    const uint32_t gp = *reinterpret_cast<const uint32_t*>(g + c);
    float* xp = x + (size_t)b * H + c;
    float2 v = *reinterpret_cast<const float2*>(xp);
    if (splits > 0) {
      float2 acc = make_float2(0.f, 0.f);
#pragma unroll 8
      for (int sp = 0; sp < splits; ++sp) {
        const float2 pv = *reinterpret_cast<const float2*>(partial + ((size_t)sp * B + b) * H + c);
        acc.x += pv.x;
        acc.y += pv.y;
      }
      v.x += acc.x;
      v.y += acc.y;
      *reinterpret_cast<float2*>(xp) = v;
    }
    sq = v.x * v.x + v.y * v.y;
    T* ap = a + (size_t)b * lda + c;
    ap[0] = from_f<T>(v.x * __uint_as_float(gp << 16));
    ap[1] = from_f<T>(v.y * __uint_as_float(gp & 0xffff0000u));
  }
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) sq += __shfl_xor(sq, o);
  if ((t & 31) == 0 && b < B) ss_out[(size_t)blockIdx.x * B + b] = sq;
}

template <typename T>
hipError_t resid_fold(const float* partial, int splits, float* x, int B, int H, const bf16_t* g, T* a, int lda,
                      float* ss_out, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (H % 64 || lda % 2 || (splits > 0 && !partial) || !ss_out) return hipErrorInvalidValue;
  hipLaunchKernelGGL((resid_fold_kernel<T>), dim3(H / 64, (B + 7) / 8), dim3(256), 0, s, partial, splits, x, B, H, g, a,
                     lda, ss_out);
  return hipGetLastError();
}

__global__ void argmax_finish_kernel(const unsigned long long* __restrict__ keys, int B, int* __restrict__ ids) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) ids[b] = (int)~(uint32_t)(keys[b] & 0xffffffffull);
}

hipError_t argmax_finish(const unsigned long long* keys, int B, int* ids, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_finish_kernel, dim3((B + 63) / 64), dim3(64), 0, s, keys, B, ids);
  return hipGetLastError();
}

// ------------------------------------------------------------------ embedding gather
template <typename T>
__global__ void embed_kernel(const T* __restrict__ vis, int n_vis, const int* __restrict__ ids, int n_ids,
                             const bf16_t* __restrict__ embed, int H, float* __restrict__ x) {
  const long total = (long)(n_vis + n_ids) * H;
  for (long idx = (long)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += (long)gridDim.x * blockDim.x) {
    const int r = (int)(idx / H), c = (int)(idx % H);
    x[idx] = r < n_vis ? to_f<T>(vis[(size_t)r * H + c]) : bf2f(embed[(size_t)ids[r - n_vis] * H + c]);
  }
}

template <typename T>
hipError_t embed_rows(const T* vis, int n_vis, const int* ids, int n_ids, const bf16_t* embed, int H, float* x,
                      hipStream_t s) {
  const long total = (long)(n_vis + n_ids) * H;
  if (total <= 0) return hipSuccess;
  const int grid = (int)std::min<long>((total + 255) / 256, 65536);
  hipLaunchKernelGGL((embed_kernel<T>), dim3(grid), dim3(256), 0, s, vis, n_vis, ids, n_ids, embed, H, x);
  return hipGetLastError();
}

// ------------------------------------------------------------------ decode step start
// One workgroup per sequence: gather the token's embedding row into the fp32 residual stream,
// write it times the first RMSNorm's gain for the first projection, and sum its squares (the
// norm's statistic, as part 0 of its per-tile parts); clear the argmax keys and tile counters.
template <typename T>
__global__ void __launch_bounds__(256) decode_embed_kernel(const int* __restrict__ ids, const bf16_t* __restrict__ embed,
                                                           int H, const bf16_t* __restrict__ g, float* __restrict__ x,
                                                           T* __restrict__ a, float* __restrict__ ss0, int ss_parts,
                                                           unsigned long long* __restrict__ keys,
                                                           unsigned* __restrict__ counters, int n_counters,
                                                           const int* __restrict__ pos, float theta, int D,
                                                           float* __restrict__ rope) {
  __shared__ float red[4];
  const int b = blockIdx.x, B = gridDim.x;
  const bf16_t* e = embed + (size_t)ids[b] * H;
  float* xr = x + (size_t)b * H;
  T* ar = a + (size_t)b * H;
  float ss = 0.f;
  for (int c = threadIdx.x; c < H; c += 256) {
    const float v = bf2f(e[c]);
    xr[c] = v;
    ar[c] = from_f<T>(v * bf2f(g[c]));
    ss += v * v;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  for (int t = 1 + threadIdx.x; t < ss_parts; t += 256) ss0[(size_t)t * B + b] = 0.f;
  if (threadIdx.x == 0) keys[b] = 0ull;
  if (b == 0)
    for (int i = threadIdx.x; i < n_counters; i += 256) counters[i] = 0u;
  // the rotary sines and cosines at this step's position, shared by every layer
  for (int c = threadIdx.x; c < D / 2; c += 256) {
    float sn, cs;
    rope_sincos(pos[b], c, D, theta, &sn, &cs);
    rope[(size_t)b * D + c] = sn;
    rope[(size_t)b * D + D / 2 + c] = cs;
  }
  __syncthreads();
  if (threadIdx.x == 0) ss0[b] = red[0] + red[1] + red[2] + red[3];
}

template <typename T>
hipError_t decode_embed(const int* ids, int B, const bf16_t* embed, int H, const bf16_t* g, float* x, T* a, float* ss0,
                        int ss_parts, unsigned long long* keys, unsigned* counters, int n_counters, const int* pos,
                        float theta, int D, float* rope, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL((decode_embed_kernel<T>), dim3(B), dim3(256), 0, s, ids, embed, H, g, x, a, ss0, ss_parts, keys,
                     counters, n_counters, pos, theta, D, rope);
  return hipGetLastError();
}
template hipError_t decode_embed<bf16_t>(const int*, int, const bf16_t*, int, const bf16_t*, float*, bf16_t*, float*, int,
                                         unsigned long long*, unsigned*, int, const int*, float, int, float*, hipStream_t);
template hipError_t decode_embed<float>(const int*, int, const bf16_t*, int, const bf16_t*, float*, float*, float*, int,
                                        unsigned long long*, unsigned*, int, const int*, float, int, float*, hipStream_t);

// ------------------------------------------------------------------ CU placement probe
__global__ void cu_probe_kernel(uint32_t* __restrict__ out, int n) {
  if (threadIdx.x == 0 && (int)blockIdx.x < n) {
    uint32_t hw, xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const uint32_t cu = (hw >> 8) & 0xfu, se = (hw >> 13) & 0x7u;
    out[blockIdx.x] = ((xcc & 0xfu) << 16) | (se << 8) | cu;
  }
  // keep each workgroup resident briefly so that the dispatcher spreads them over all CUs
  const long long t0 = clock64();
  while (clock64() - t0 < 20000) {
  }
}

hipError_t cu_probe(hipStream_t s, uint32_t* out, int n) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(cu_probe_kernel, dim3(n), dim3(64), 0, s, out, n);
  return hipGetLastError();
}

// ------------------------------------------------------------------ greedy argmax (ties -> lowest index)
__global__ void argmax_kernel(const float* __restrict__ logits, int V, int* __restrict__ out) {
  const float* row = logits + (size_t)blockIdx.x * V;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  for (int i = threadIdx.x; i < V; i += blockDim.x) {
    const float v = row[i];
    if (v > best) { best = v; bi = i; }   // strided scan: first hit per thread is its lowest index
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(best, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
  }
  __shared__ float sv[16];
  __shared__ int si[16];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { sv[w] = best; si[w] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int j = 1; j < (int)(blockDim.x >> 6); ++j)
      if (sv[j] > best || (sv[j] == best && si[j] < bi)) { best = sv[j]; bi = si[j]; }
    out[blockIdx.x] = bi;
  }
}

hipError_t argmax_rows(const float* logits, int B, int V, int* out, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(B), dim3(1024), 0, s, logits, V, out);
  return hipGetLastError();
}

template hipError_t norm_rows<bf16_t>(const float*, int, int, const bf16_t*, const bf16_t*, float, int, bf16_t*, int, int, int, int, hipStream_t);
template hipError_t norm_rows<float>(const float*, int, int, const bf16_t*, const bf16_t*, float, int, float*, int, int, int, int, hipStream_t);
template hipError_t split_norm_rows<bf16_t>(const float*, int, size_t, float*, int, int, const bf16_t*, const bf16_t*, float, int,
                                            bf16_t*, int, hipStream_t);
template hipError_t split_norm_rows<float>(const float*, int, size_t, float*, int, int, const bf16_t*, const bf16_t*, float, int,
                                           float*, int, hipStream_t);
template hipError_t patchify<bf16_t>(const bf16_t*, int, int, int, int, int, bf16_t*, hipStream_t);
template hipError_t patchify<float>(const bf16_t*, int, int, int, int, int, float*, hipStream_t);
template <typename T>
__global__ void zero_tail_cols_kernel(T* __restrict__ buf, long rows, int ld, int c0) {
  const int w = ld - c0;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < rows * w; i += (long)gridDim.x * blockDim.x)
    buf[(i / w) * ld + c0 + i % w] = T(0);
}

template <typename T>
hipError_t zero_tail_cols(T* buf, long rows, int ld, int c0, hipStream_t s) {
  if (rows <= 0 || c0 >= ld) return hipSuccess;
  const long n = rows * (ld - c0);
  hipLaunchKernelGGL((zero_tail_cols_kernel<T>), dim3((unsigned)std::min<long>((n + 255) / 256, 4096)), dim3(256), 0, s,
                     buf, rows, ld, c0);
  return hipGetLastError();
}
template hipError_t zero_tail_cols<bf16_t>(bf16_t*, long, int, int, hipStream_t);
template hipError_t zero_tail_cols<float>(float*, long, int, int, hipStream_t);

template hipError_t qkv_prefill<bf16_t>(bf16_t*, int, int, int, int, int, float, int, bf16_t*, int, bf16_t*, bf16_t*, const int*, int, hipStream_t, unsigned*, int);
template hipError_t qkv_prefill<float>(float*, int, int, int, int, int, float, int, float*, int, float*, float*, const int*, int, hipStream_t, unsigned*, int);
template hipError_t resid_rmsnorm<bf16_t>(const float*, int, float*, int, int, const bf16_t*, float, bf16_t*, int, unsigned long long*, hipStream_t);
template hipError_t resid_rmsnorm<float>(const float*, int, float*, int, int, const bf16_t*, float, float*, int, unsigned long long*, hipStream_t);
template hipError_t resid_fold<bf16_t>(const float*, int, float*, int, int, const bf16_t*, bf16_t*, int, float*,
                                       hipStream_t);
template hipError_t resid_fold<float>(const float*, int, float*, int, int, const bf16_t*, float*, int, float*, hipStream_t);
template hipError_t embed_rows<bf16_t>(const bf16_t*, int, const int*, int, const bf16_t*, int, float*, hipStream_t);
template hipError_t embed_rows<float>(const float*, int, const int*, int, const bf16_t*, int, float*, hipStream_t);

}  // namespace nova
