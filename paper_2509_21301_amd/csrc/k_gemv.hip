// Thin GEMM for the decode linears and the LM head: Y[B,N] = X[B,K] W[N,K]^T, B <= 32.
//
// Decode is bound by streaming the weights from HBM (the paper's Table 3 decode row and
// Sec. 3.2.1).  Each wave owns 16 weight rows and walks K in 256-wide chunks.  A chunk is read
// with eight 16-byte-per-lane loads, each covering two whole rows (2 x 512 contiguous bytes):
// loads that touch only part of a cache line per row cost far more per byte on a CU, which shows
// most when the stream runs on a fraction of the chip.  The chunk then passes through a
// wave-private LDS tile into the MFMA 16x16x32 operand layout (row = lane % 16), with an XOR
// swizzle that keeps both the writes and the reads free of bank conflicts.  The batch is the
// other MFMA operand: X chunks stream through a two-slot LDS ring shared by the workgroup's four
// waves, one barrier per chunk.  Weight and X loads run two chunks ahead in registers, issued in
// the order they are consumed so that each wait covers only its own chunk.
// When N alone gives too few workgroups, K is split and a small second pass reduces the fp32
// partials and applies the epilogue; otherwise the epilogue is applied directly.
// RMSNorm folding (small decode batches): a residual producer (O, down projection) writes the
// updated residual x, x times the next norm's gain, and per-64-row-tile sums of squares of x;
// with split-K the last split of each tile (a device-scope arrival counter; partials written
// through to the coherent level, so no cache write-back is needed) folds the partials in.  The
// consumer (QKV, gate/up, LM head) reads x * gain as X and scales output column b by
// rsqrt(mean x_b^2 + eps), summing the tile parts in a fixed order.
// The k index of an MFMA fragment only has to agree between its two operands, which leaves the
// assignment of k pieces to lanes free.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace nova {

constexpr int GV_KC = 256;             // K chunk per pipeline step (32 pieces of 8)
constexpr int GV_RW = 16;              // weight rows per wave
constexpr int GV_ROWS = 4 * GV_RW;     // rows per workgroup (4 waves)
constexpr int GV_MAX_SPLITS = 16;

// K splits: as many as keep the workgroups (64 rows each) within the stream's compute units, one
// workgroup per CU.  Measured on the decode shapes at 64, 128 and 256 CUs, a CU streams one
// workgroup's rows at a good rate, while a second round of workgroups on some CUs leaves the
// others idle at the end (the down projection at batch 1 on 256 CUs: 27.4 us with 224
// workgroups, 29.9-35.5 us with 280 to 560).  Each split is a run of whole 256-wide chunks, and
// no split is empty.
int gemv_splits(int N, int K, int B, bool f32x, int cus) {
  (void)B;
  (void)f32x;
  const int chunks = K / GV_KC, wgs = N / GV_ROWS;
  int s = wgs >= cus ? 1 : std::min(cus / wgs, GV_MAX_SPLITS);
  s = std::max(1, std::min(s, chunks));
  const int per = (chunks + s - 1) / s;          // chunks per split
  return (chunks + per - 1) / per;
}

size_t gemv_partial_floats(int B, int N, int K, bool f32x, int cus) {
  const int s = gemv_splits(N, K, B, f32x, cus);
  return s > 1 ? (size_t)s * B * N : 0;
}

// Element (row, k) of a 256-wide tile with rows of 32 16-byte pieces: piece k/8 is stored at
// slot (k/8) ^ (row % 16).
__device__ __forceinline__ int swz(int row, int piece) { return row * GV_KC + 8 * (piece ^ (row & 15)); }

// TA: activation type of X (bf16, or fp32 for the exact mode whose operands are split into bf16
// hi + lo).  NSCALE: X holds x * gain of a folded RMSNorm; output columns are scaled by the row's
// rsqrt(mean x^2 + eps), from the producer's per-tile sums of squares.
template <typename TA, typename OT, int NB, int EPI, bool DIRECT, bool NSCALE>
__global__ void __launch_bounds__(256) gemv_kernel(GemvArgs p, int kc) {
  using TX = TA;
  constexpr bool F32X = sizeof(TA) == 4;                  // X fp32, operands split into bf16 hi + lo
  constexpr int XROWS = 16 * NB;                          // batch rows held (B padded)
  constexpr int XR = F32X ? 1 : 2;                        // X ring slots
  constexpr int XSLOT = XROWS * GV_KC * (F32X ? 2 : 1);   // bf16 per slot (fp32 mode: hi, lo)
  constexpr int XPT = XROWS / 8;                          // 16-byte X pieces per thread per chunk
  constexpr int XL = F32X ? 2 * XPT : XPT;                // X loads per thread per chunk
  __shared__ __align__(16) bf16_t wt[4][GV_RW * GV_KC];
  __shared__ __align__(16) bf16_t xs[XR * XSLOT];
  __shared__ float red[EPI == EPI_RESID ? 4 : 1][32];     // per-wave row statistics (residual producers)
  __shared__ float rstd_s[NSCALE ? 32 : 1];                // per-row RMSNorm scale (normalising consumers)
  __shared__ unsigned long long am_s[EPI == EPI_ARGMAX ? 4 : 1][16];   // per-wave argmax keys

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_base = blockIdx.x * GV_ROWS + wave * GV_RW;
  const int split = blockIdx.y;
  const int k_begin = split * kc, k_end = min(k_begin + kc, p.K);
  const int nchunks = (k_end - k_begin) / GV_KC;
  const int n = lane & 15, g = lane >> 4;          // MFMA operand row and k group
  const int h = lane >> 5, pc = lane & 31;         // load row within a pair, piece

  // weight load i of a chunk: rows 2i + h, piece pc (lanes 0-31 and 32-63 each read one row)
  const bf16_t* wsrc = p.W + (size_t)(n_base + h) * p.ldw + k_begin + 8 * pc;
  typedef u32x4 WBuf[8];
  auto load_w = [&](int c, WBuf& w) {
    const bf16_t* src = wsrc + (size_t)min(c, nchunks - 1) * GV_KC;   // tail: re-read the last chunk
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = *reinterpret_cast<const u32x4*>(src + (size_t)(2 * i) * p.ldw);
  };
  // X piece q of a chunk for this thread: batch row tid / 32 + 8q (clamped to B-1: those rows
  // only feed output columns that are never stored), piece tid % 32
  const TX* X = reinterpret_cast<const TX*>(p.X);
  typedef u32x4 XBuf[XL];
  auto load_x = [&](int c, XBuf& x) {
    const int k = k_begin + min(c, nchunks - 1) * GV_KC + 8 * pc;
#pragma unroll
    for (int q = 0; q < XPT; ++q) {
      const TX* src = X + (size_t)min((tid >> 5) + 8 * q, p.B - 1) * p.ldx + k;
      if constexpr (F32X) {
        x[2 * q] = *reinterpret_cast<const u32x4*>(src);
        x[2 * q + 1] = *reinterpret_cast<const u32x4*>(src + 4);
      } else {
        x[q] = *reinterpret_cast<const u32x4*>(src);
      }
    }
  };
  auto store_x = [&](const XBuf& x, int slot) {
    bf16_t* dst = xs + slot * XSLOT;
#pragma unroll
    for (int q = 0; q < XPT; ++q) {
      const int r = (tid >> 5) + 8 * q;
      if constexpr (F32X) {
        float x8[8];
        *reinterpret_cast<u32x4*>(x8) = x[2 * q];
        *reinterpret_cast<u32x4*>(x8 + 4) = x[2 * q + 1];
        Frag8 hi, lo;
        split8(x8, hi, lo);
        *reinterpret_cast<Frag8*>(dst + swz(r, pc)) = hi;
        *reinterpret_cast<Frag8*>(dst + XROWS * GV_KC + swz(r, pc)) = lo;
      } else {
        *reinterpret_cast<u32x4*>(dst + swz(r, pc)) = x[q];
      }
    }
  };

  f32x4 acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16_t* tw = wt[wave];

  // one chunk: weights through the wave's tile into operand layout, then MFMAs against the X slot;
  // MFMA u takes piece 4u + g of row n from both operands
  auto compute = [&](int c, const WBuf& w) {
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4*>(tw + swz(2 * i + h, pc)) = w[i];
    // a wave's LDS operations execute in order; only the compiler has to be kept from moving
    // the reads above the writes (or the next chunk's writes above these reads)
    asm volatile("" ::: "memory");
    const bf16_t* xb = xs + (c % XR) * XSLOT;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const Frag8 wf = *reinterpret_cast<const Frag8*>(tw + swz(n, 4 * u + g));
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const Frag8 xf = *reinterpret_cast<const Frag8*>(xb + swz(16 * j + n, 4 * u + g));
        acc[j] = mfma16(wf, xf, acc[j]);
        if constexpr (F32X) {
          const Frag8 xl = *reinterpret_cast<const Frag8*>(xb + XROWS * GV_KC + swz(16 * j + n, 4 * u + g));
          acc[j] = mfma16(wf, xl, acc[j]);
        }
      }
    }
    asm volatile("" ::: "memory");
  };
  // compute chunk c, then publish X(c+1) in its ring slot (with one slot, only after every wave
  // is done with chunk c); the barrier makes it visible and frees the other slot
  auto step = [&](int c, const WBuf& w, const XBuf& xnext) {
    compute(c, w);
    if (c + 1 < nchunks) {
      if constexpr (XR == 1) __syncthreads();
      store_x(xnext, (c + 1) % XR);
    }
    __syncthreads();
  };

  // loads are unconditional (clamped at the tail) and issued in consumption order, so that the
  // wait before each use covers only its own chunk
  // the row statistic first (ahead of the weight stream in the in-order load counter): wave w
  // takes batch rows w, w + 4, ...; lane t holds tile part t (<= 64 parts), summed by a
  // fixed-order butterfly
  float ssv[NSCALE ? (16 * NB + 3) / 4 : 1];
  if constexpr (NSCALE) {
#pragma unroll
    for (int i = 0; i < (16 * NB + 3) / 4; ++i) {
      const int b = min(wave + 4 * i, p.B - 1);
      ssv[i] = lane < p.ss_parts ? p.ss_in[(size_t)lane * p.B + b] : 0.f;
    }
  }
  WBuf w0, w1, w2;
  XBuf x0, x1, x2;
  load_x(0, x0);
  load_w(0, w0);
  load_x(1, x1);
  load_w(1, w1);
  if constexpr (NSCALE) {
#pragma unroll
    for (int i = 0; i < (16 * NB + 3) / 4; ++i) {
      const float ss = wave_sum(ssv[i]);
      if (lane == 0 && wave + 4 * i < p.B) rstd_s[wave + 4 * i] = rsqrtf(ss / p.K + p.eps);
    }
  }
  store_x(x0, 0);
  __syncthreads();
  for (int c = 0; c < nchunks; c += 3) {
    load_x(c + 2, x2);
    load_w(c + 2, w2);
    step(c, w0, x1);
    load_x(c + 3, x0);
    load_w(c + 3, w0);
    if (c + 1 < nchunks) step(c + 1, w1, x2);
    load_x(c + 4, x1);
    load_w(c + 4, w1);
    if (c + 2 < nchunks) step(c + 2, w2, x0);
  }

  // lane holds D[n = 4*(lane/16) + r][b = lane%16] of each 16x16 tile
  if constexpr (NSCALE) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const float rstd = rstd_s[min(j * 16 + (lane & 15), p.B - 1)];
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[j][r] *= rstd;
    }
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int b = j * 16 + (lane & 15);
    if constexpr (EPI == EPI_ARGMAX && DIRECT) {
      // greedy argmax fused into the LM head: best (logit, lowest id) of the lane's 4 rows, then
      // of the 16 rows of the tile (lanes 16 apart), merged across workgroups by a 64-bit
      // atomic max on (order-preserving logit bits, ~id)
      unsigned long long key = 0ull;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int nr = n_base + (lane >> 4) * 4 + r;
        const float v = acc[j][r];
        if (p.out != nullptr && b < p.B) reinterpret_cast<float*>(p.out)[(size_t)b * p.ldo + nr] = v;
        const uint32_t u = __float_as_uint(v);
        const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
        const unsigned long long k = ((unsigned long long)ord << 32) | (uint32_t)~(uint32_t)nr;
        key = k > key ? k : key;
      }
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const unsigned long long other = __shfl_xor(key, o, 64);
        key = other > key ? other : key;
      }
      // the workgroup's 4 waves combine through LDS, and one lane per row merges the result only
      // if it beats the row's best so far (which only grows, so a stale read merely costs an
      // extra atomic): some 2400 workgroups of the LM head would otherwise queue 4 atomics each
      // on the same address (a fifth of the head's time)
      if (lane < 16) am_s[wave][lane] = key;
      __syncthreads();
      if (wave == 0 && lane < 16 && b < p.B) {
        unsigned long long k = am_s[0][lane];
#pragma unroll
        for (int w = 1; w < 4; ++w) k = am_s[w][lane] > k ? am_s[w][lane] : k;
        if (k > __hip_atomic_load(p.argmax_keys + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
          atomicMax(p.argmax_keys + b, k);
      }
      __syncthreads();          // am_s is reused by the next column group
      continue;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int nr = (lane >> 4) * 4 + r;
      if constexpr (!DIRECT) {
        float* dst = p.partial + ((size_t)split * p.B + b) * p.N + n_base + nr;
        if (EPI == EPI_RESID && p.counters != nullptr) {
          // written through to the device-coherent level: the tile's last split reads them
          if (b < p.B) __hip_atomic_store(dst, acc[j][r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
          if (b < p.B) *dst = acc[j][r];
        }
      } else if constexpr (EPI == EPI_SWIGLU) {
        // rows interleaved in blocks of 8: rows 0-7 of the tile are gate rows, 8-15 the matching
        // up rows, held by lanes 32 apart
        const float up = __shfl_xor(acc[j][r], 32, 64);
        if (lane < 32 && b < p.B) {
          const int oc = (n_base >> 1) + nr;
          reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + oc] = from_f<OT>(silu(acc[j][r]) * up);
        }
      } else if constexpr (EPI == EPI_RESID) {
        if (b < p.B) {
          float* o = reinterpret_cast<float*>(p.out) + (size_t)b * p.ldo + n_base + nr;
          const float xn = *o + acc[j][r];
          *o = xn;
          if (p.gain_out != nullptr)
            reinterpret_cast<TA*>(p.aout)[(size_t)b * p.ldao + n_base + nr] = from_f<TA>(xn * bf2f(p.gain_out[n_base + nr]));
          acc[j][r] = xn * xn;         // kept for the row statistic below
        } else {
          acc[j][r] = 0.f;
        }
      } else {
        if (b < p.B) reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + n_base + nr] = from_f<OT>(acc[j][r]);
      }
    }
    if constexpr (EPI == EPI_RESID && DIRECT) {
      // this wave's 16 rows of the updated residual, summed per batch row (lanes 16 apart share b)
      float sq = acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
      sq += __shfl_xor(sq, 16, 64);
      sq += __shfl_xor(sq, 32, 64);
      if (lane < 16) red[wave][j * 16 + lane] = sq;
    }
  }
  if constexpr (EPI == EPI_RESID && DIRECT) {
    if (p.ss_out != nullptr) {       // the workgroup's 64 rows: the 4 waves in a fixed order
      __syncthreads();
      if (tid < p.B) p.ss_out[(size_t)blockIdx.x * p.B + tid] = red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid];
    }
  }
  if constexpr (EPI == EPI_RESID && !DIRECT) {
    if (p.counters != nullptr) {
      // the last split to finish this workgroup's 64 rows folds every split's partials into the
      // residual and writes the rows' sum of squares.  The partials are device-scope atomic
      // stores, written through to the coherent level; every thread waits until its stores are
      // acknowledged there (s_waitcnt) before the workgroup barrier, and only then does thread 0
      // increment the device-scope counter, so a split's partials are at the coherent level
      // before its arrival is; the last split to arrive reads them back with device-scope
      // atomic loads from that level.  The counter is relaxed: at device scope a release /
      // acquire increment would also write back and invalidate the XCD's L2 in every
      // workgroup (buffer_wbl2 / buffer_inv), which measured 3.6% and 7% slower decode steps at
      // batch 1 and 8, for data that never sits in a non-coherent cache line.
      __shared__ int last;
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0)
        last = __hip_atomic_fetch_add(p.counters + blockIdx.x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               gridDim.y - 1;
      __syncthreads();
      if (!last) return;
      float* xo = reinterpret_cast<float*>(p.out);
      const int n0 = blockIdx.x * GV_ROWS;
      const float gn = p.gain_out != nullptr ? bf2f(p.gain_out[n0 + lane]) : 0.f;
      // wave w takes batch rows w, w + 4, ... (at most 8); lane = row within the tile.  Each load is
      // a round trip to the coherent level, so the loads of 8 splits are all issued before any is
      // summed (then summed in split order)
      constexpr int BPW = (16 * NB + 3) / 4;
      float v[BPW];
#pragma unroll
      for (int i = 0; i < BPW; ++i) v[i] = 0.f;
      for (int sp0 = 0; sp0 < (int)gridDim.y; sp0 += 8) {
        float t[8][BPW];
#pragma unroll
        for (int k = 0; k < 8; ++k)
#pragma unroll
          for (int i = 0; i < BPW; ++i) {
            const int b = wave + 4 * i, sp = sp0 + k;
            t[k][i] = b < p.B && sp < (int)gridDim.y
                          ? __hip_atomic_load(p.partial + ((size_t)sp * p.B + b) * p.N + n0 + lane, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT)
                          : 0.f;
          }
#pragma unroll
        for (int k = 0; k < 8; ++k)
#pragma unroll
          for (int i = 0; i < BPW; ++i)
            if (sp0 + k < (int)gridDim.y) v[i] += t[k][i];
      }
#pragma unroll
      for (int i = 0; i < BPW; ++i) {
        const int b = wave + 4 * i;
        if (b >= p.B) break;             // uniform per wave
        float* o = xo + (size_t)b * p.ldo + n0 + lane;
        const float xn = *o + v[i];
        *o = xn;
        if (p.gain_out != nullptr) reinterpret_cast<TA*>(p.aout)[(size_t)b * p.ldao + n0 + lane] = from_f<TA>(xn * gn);
        const float sq = wave_sum(xn * xn);
        if (lane == 0 && p.ss_out != nullptr) p.ss_out[(size_t)blockIdx.x * p.B + b] = sq;
      }
      if (tid == 0) __hip_atomic_store(p.counters + blockIdx.x, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Sum the split partials and apply the epilogue: one thread per output element.
template <typename OT, int EPI>
__global__ void gemv_reduce(GemvArgs p, int splits) {
  const int ncols = EPI == EPI_SWIGLU ? p.N / 2 : p.N;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const bool live = idx < (long)p.B * ncols;
  const int b = live ? (int)(idx / ncols) : 0, c = live ? (int)(idx % ncols) : 0;
  auto sum = [&](int n) {
    float v = 0.f;
#pragma unroll 4
    for (int s = 0; s < splits; ++s) v += p.partial[((size_t)s * p.B + b) * p.N + n];
    return v;
  };
  if constexpr (EPI == EPI_ARGMAX) {
    // logits of one row are contiguous and ncols is a multiple of 64, so a wave shares one b
    const float v = live ? sum(c) : -INFINITY;
    if (live && p.out != nullptr) reinterpret_cast<float*>(p.out)[(size_t)b * p.ldo + c] = v;
    const uint32_t u = __float_as_uint(v);
    const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    unsigned long long key = live ? (((unsigned long long)ord << 32) | (uint32_t)~(uint32_t)c) : 0ull;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const unsigned long long other = __shfl_xor(key, o, 64);
      key = other > key ? other : key;
    }
    if ((threadIdx.x & 63) == 0 && key != 0ull) atomicMax(p.argmax_keys + b, key);
    return;
  }
  if (!live) return;
  if constexpr (EPI == EPI_SWIGLU) {
    const int n = (c >> 3) * 16 + (c & 7);     // gate row; its up row is 8 further
    reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + c] = from_f<OT>(silu(sum(n)) * sum(n + 8));
  } else if constexpr (EPI == EPI_RESID) {
    reinterpret_cast<float*>(p.out)[(size_t)b * p.ldo + c] += sum(c);
  } else {
    reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + c] = from_f<OT>(sum(c));
  }
}

template <typename TA, typename OT, int NB, int EPI, bool NSCALE>
static hipError_t gemv_launch(const GemvArgs& p, hipStream_t s) {
  constexpr bool F32X = sizeof(TA) == 4;
  const int splits = gemv_splits(p.N, p.K, p.B, F32X, p.cus);
  const int chunks = p.K / GV_KC;
  const int kc = (chunks + splits - 1) / splits * GV_KC;
  dim3 grid(p.N / GV_ROWS, splits);
  if (splits == 1) {
    hipLaunchKernelGGL((gemv_kernel<TA, OT, NB, EPI, true, NSCALE>), grid, dim3(256), 0, s, p, kc);
    return hipGetLastError();
  }
  if (!p.partial || (EPI == EPI_RESID && p.ss_out != nullptr && p.counters == nullptr)) return hipErrorInvalidValue;
  hipLaunchKernelGGL((gemv_kernel<TA, OT, NB, EPI, false, NSCALE>), grid, dim3(256), 0, s, p, kc);
  hipError_t e = hipGetLastError();
  // out == null (except for the argmax, whose logits are optional): the caller reduces the
  // partials; a residual producer with tile counters has folded them in already
  if (e != hipSuccess || (p.out == nullptr && EPI != EPI_ARGMAX)) return e;
  if (EPI == EPI_RESID && p.counters != nullptr) return e;
  const long n = (long)p.B * (EPI == EPI_SWIGLU ? p.N / 2 : p.N);
  hipLaunchKernelGGL((gemv_reduce<OT, EPI>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, splits);
  return hipGetLastError();
}

template <typename TX, typename OT>
hipError_t gemv(const GemvArgs& p, int epi, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.B > 32 || p.N % GV_ROWS || p.K <= 0 || p.K % GV_KC || p.ldx % 8 || p.ldw % 8 || p.cus <= 0) return hipErrorInvalidValue;
  if (epi == EPI_ARGMAX && (!p.argmax_keys || p.N % 64)) return hipErrorInvalidValue;
  if (p.ss_in != nullptr && (p.ss_parts <= 0 || p.ss_parts > 64)) return hipErrorInvalidValue;
  if ((p.ss_out != nullptr || p.counters != nullptr || p.gain_out != nullptr) && (epi != EPI_RESID || p.out == nullptr))
    return hipErrorInvalidValue;
  if (p.gain_out != nullptr && p.aout == nullptr) return hipErrorInvalidValue;
  const bool two = p.B > 16, norm = p.ss_in != nullptr;
#define NOVA_GEMV_CASE(E)                                                                                 \
  case E:                                                                                                 \
    if (norm) return two ? gemv_launch<TX, OT, 2, E, true>(p, s) : gemv_launch<TX, OT, 1, E, true>(p, s); \
    return two ? gemv_launch<TX, OT, 2, E, false>(p, s) : gemv_launch<TX, OT, 1, E, false>(p, s);
  switch (epi) {
    NOVA_GEMV_CASE(EPI_STORE)
    NOVA_GEMV_CASE(EPI_RESID)
    NOVA_GEMV_CASE(EPI_SWIGLU)
    NOVA_GEMV_CASE(EPI_ARGMAX)
  }
#undef NOVA_GEMV_CASE
  return hipErrorInvalidValue;
}

// Decode linear on the vector ALUs: one wave per output row n.  Lane l takes the 16-byte pieces
// k = 8 l + 512 i of the weight row (each load instruction covers 1 KB of contiguous weights) and
// the same pieces of the B input rows, accumulates in fp32 with fused multiply-adds, and the
// wave sums the lanes.  No LDS and about 40 registers, so its waves fit beside another kernel's
// workgroups on the same compute unit.
template <int NB>
__global__ void __launch_bounds__(256) gemv_valu_kernel(const bf16_t* __restrict__ X, int ldx, const bf16_t* __restrict__ W,
                                                        int ldw, int N, int K, float* __restrict__ out, int ldo) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const bf16_t* wr = W + (size_t)n * ldw;
  float acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = 0.f;
#pragma unroll 7
  for (int k0 = lane * 8; k0 < K; k0 += 512) {
    const u32x4 wv = *reinterpret_cast<const u32x4*>(wr + k0);
    float wf[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      wf[2 * e] = __uint_as_float(wv[e] << 16);
      wf[2 * e + 1] = __uint_as_float(wv[e] & 0xffff0000u);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const u32x4 xv = *reinterpret_cast<const u32x4*>(X + (size_t)b * ldx + k0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[b] = fmaf(wf[2 * e], __uint_as_float(xv[e] << 16), acc[b]);
        acc[b] = fmaf(wf[2 * e + 1], __uint_as_float(xv[e] & 0xffff0000u), acc[b]);
      }
    }
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = wave_sum(acc[b]);
  if (lane < NB) {
    float v = acc[0];
#pragma unroll
    for (int b = 1; b < NB; ++b) v = lane == b ? acc[b] : v;
    out[(size_t)lane * ldo + n] += v;
  }
}

hipError_t gemv_valu(const bf16_t* X, int ldx, const bf16_t* W, int ldw, int B, int N, int K, float* out, int ldo,
                     hipStream_t s) {
  if (B <= 0 || N <= 0) return hipSuccess;
  if (B > 4 || K <= 0 || K % 512 || ldx % 8 || ldw % 8) return hipErrorInvalidValue;
  const dim3 grid((N + 3) / 4);
  switch (B) {
    case 1: hipLaunchKernelGGL((gemv_valu_kernel<1>), grid, dim3(256), 0, s, X, ldx, W, ldw, N, K, out, ldo); break;
    case 2: hipLaunchKernelGGL((gemv_valu_kernel<2>), grid, dim3(256), 0, s, X, ldx, W, ldw, N, K, out, ldo); break;
    case 3: hipLaunchKernelGGL((gemv_valu_kernel<3>), grid, dim3(256), 0, s, X, ldx, W, ldw, N, K, out, ldo); break;
    default: hipLaunchKernelGGL((gemv_valu_kernel<4>), grid, dim3(256), 0, s, X, ldx, W, ldw, N, K, out, ldo); break;
  }
  return hipGetLastError();
}

template hipError_t gemv<bf16_t, bf16_t>(const GemvArgs&, int, hipStream_t);
template hipError_t gemv<bf16_t, float>(const GemvArgs&, int, hipStream_t);
template hipError_t gemv<float, float>(const GemvArgs&, int, hipStream_t);

}  // namespace nova
