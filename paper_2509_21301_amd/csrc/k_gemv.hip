// Thin GEMM for the decode linears and the LM head: Y[B,N] = X[B,K] W[N,K]^T, B <= 32.
//
// Decode is bound by streaming the weights from HBM (the paper's Table 3 decode row and
// Sec. 3.2.1).  Each wave streams 32 weight rows with 16-byte loads (16 per lane per 256-wide
// K chunk, 32 in flight with the prefetch), and feeds them to MFMA 16x16x32 as
// the A operand with the batch as the 16-wide B operand (a second MFMA covers rows 16..31 of
// the batch).  X fragments come straight from L2 (X is small and shared by every workgroup);
// weight loads run one chunk ahead of the MFMAs, with no LDS and no barriers.  When N alone
// gives too few workgroups, K is split and a small second pass reduces the fp32 partials and applies the
// epilogue; otherwise the epilogue is applied directly.
// The k index of an MFMA fragment only has to agree between its A and B operands, which leaves
// the assignment of k pieces to lanes free; it is chosen for coalescing.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace nova {

constexpr int GV_KC = 256;          // K chunk per pipeline step

constexpr int GV_RW = 16;           // weight rows per wave
constexpr int GV_MAX_SPLITS = 16;

// K splits so that the launch has about 2048 waves (every CU holding several); a split is a
// run of whole 256-wide chunks, the last one possibly shorter.
int gemv_splits(int N, int K) {
  const int chunks = K / GV_KC, waves = N / GV_RW;
  if (waves >= 2048) return 1;
  int s = std::min((2048 + waves - 1) / waves, GV_MAX_SPLITS);
  s = std::min(s, chunks);
  const int per = (chunks + s - 1) / s;          // chunks per split
  return (chunks + per - 1) / per;               // no empty split
}

size_t gemv_partial_floats(int B, int N, int K) {
  const int s = gemv_splits(N, K);
  return s > 1 ? (size_t)s * B * N : 0;
}

template <typename TX, typename OT, int NB, int EPI, bool DIRECT, int RW>
__global__ void __launch_bounds__(256) gemv_kernel(GemvArgs p, int kc) {
  constexpr bool F32X = sizeof(TX) == 4;
  constexpr int RG = RW / 16;                  // 16-row MFMA groups per wave
  constexpr int XN = F32X ? 2 : 1;             // 16-byte pieces per X fragment
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_base = blockIdx.x * (4 * RW) + wave * RW;
  const int split = blockIdx.y;
  const int k_begin = split * kc, k_end = min(k_begin + kc, p.K);
  const int row = lane & 15, g = lane >> 4;
  // Fragment u of a 256-wide chunk holds k = k0 + 8 * (4u + g) .. +8: the four lanes of a row
  // read 64 adjacent bytes per instruction and two instructions complete each 128-byte line.
  const bf16_t* wrow = p.W + (size_t)(n_base + row) * p.ldw + 8 * g;
  const TX* X = reinterpret_cast<const TX*>(p.X);

  f32x4 acc[RG][NB];
#pragma unroll
  for (int i = 0; i < RG; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  typedef u32x4 WBuf[RG][8];
  typedef u32x4 XBuf[NB][8][XN];
  auto load = [&](int k0, WBuf& w, XBuf& x) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int i = 0; i < RG; ++i) w[i][u] = *reinterpret_cast<const u32x4*>(wrow + (size_t)16 * i * p.ldw + k0 + 32 * u);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int b = j * 16 + row;
      const u32x4* xr = reinterpret_cast<const u32x4*>(X + (size_t)b * p.ldx + k0 + 8 * g);
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int h = 0; h < XN; ++h) x[j][u][h] = b < p.B ? xr[(32 * u) / (8 / XN) + h] : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto compute = [&](const WBuf& w, const XBuf& x) {
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        Frag8 fx, fl;
        if constexpr (F32X) {
          float x8[8];
          *reinterpret_cast<u32x4*>(x8) = x[j][u][0];
          *reinterpret_cast<u32x4*>(x8 + 4) = x[j][u][XN - 1];
          split8(x8, fx, fl);
        } else {
          fx = __builtin_bit_cast(Frag8, x[j][u][0]);
        }
#pragma unroll
        for (int i = 0; i < RG; ++i) {
          acc[i][j] = mfma16(__builtin_bit_cast(Frag8, w[i][u]), fx, acc[i][j]);
          if constexpr (F32X) acc[i][j] = mfma16(__builtin_bit_cast(Frag8, w[i][u]), fl, acc[i][j]);
        }
      }
  };

  // double buffer: chunk c+1's weights and activations are in flight while chunk c computes
  WBuf w0, w1;
  XBuf x0, x1;
  load(k_begin, w0, x0);
  for (int k0 = k_begin; k0 < k_end; k0 += 2 * GV_KC) {
    const bool has1 = k0 + GV_KC < k_end;
    if (has1) load(k0 + GV_KC, w1, x1);
    compute(w0, x0);
    if (!has1) break;
    if (k0 + 2 * GV_KC < k_end) load(k0 + 2 * GV_KC, w0, x0);
    compute(w1, x1);
  }

  // lane holds D[n = 4*(lane/16) + r][b = lane%16] of each 16x16 tile
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int b = j * 16 + (lane & 15);
    if constexpr (EPI == EPI_ARGMAX) {
      // greedy argmax fused into the LM head: best (logit, lowest id) of the lane's 4 rows, then
      // of the 16 rows of the tile (lanes 16 apart), merged across workgroups by a 64-bit
      // atomic max on (order-preserving logit bits, ~id)
      unsigned long long key = 0ull;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = n_base + (lane >> 4) * 4 + r;
        const float v = acc[0][j][r];
        if (DIRECT && p.out != nullptr && b < p.B) reinterpret_cast<float*>(p.out)[(size_t)b * p.ldo + n] = v;
        const uint32_t u = __float_as_uint(v);
        const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
        const unsigned long long k = ((unsigned long long)ord << 32) | (uint32_t)~(uint32_t)n;
        key = k > key ? k : key;
      }
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const unsigned long long other = __shfl_xor(key, o, 64);
        key = other > key ? other : key;
      }
      if (lane < 16 && b < p.B) atomicMax(p.argmax_keys + b, key);
      continue;
    }
    if constexpr (EPI == EPI_SWIGLU) {
      if (j * 16 >= p.B) continue;    // whole column group empty (uniform across the wave)
    } else {
      if (b >= p.B) continue;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int nr = (lane >> 4) * 4 + r;
      if constexpr (!DIRECT) {
        float* part = p.partial + ((size_t)split * p.B + b) * p.N;
#pragma unroll
        for (int i = 0; i < RG; ++i) part[n_base + 16 * i + nr] = acc[i][j][r];
      } else if constexpr (EPI == EPI_SWIGLU) {
        if (b >= p.B) continue;
        // rows interleaved in blocks of 8: rows 0-7 of the tile are gate rows, 8-15 the matching
        // up rows, held by lanes 32 apart
        const float gte = acc[0][j][r], up = __shfl_xor(acc[0][j][r], 32, 64);
        if (lane < 32) {
          const int oc = (n_base >> 1) + nr;
          reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + oc] = from_f<OT>(silu(gte) * up);
        }
      } else if constexpr (EPI == EPI_RESID) {
        float* o = reinterpret_cast<float*>(p.out) + (size_t)b * p.ldo;
#pragma unroll
        for (int i = 0; i < RG; ++i) o[n_base + 16 * i + nr] += acc[i][j][r];
      } else {
        OT* o = reinterpret_cast<OT*>(p.out) + (size_t)b * p.ldo;
#pragma unroll
        for (int i = 0; i < RG; ++i) o[n_base + 16 * i + nr] = from_f<OT>(acc[i][j][r]);
      }
    }
  }
}

// Sum the split partials and apply the epilogue: one thread per output element.
template <typename OT, int EPI>
__global__ void gemv_reduce(GemvArgs p, int splits) {
  const int ncols = EPI == EPI_SWIGLU ? p.N / 2 : p.N;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)p.B * ncols) return;
  const int b = (int)(idx / ncols), c = (int)(idx % ncols);
  auto sum = [&](int n) {
    float v = 0.f;
#pragma unroll 4
    for (int s = 0; s < splits; ++s) v += p.partial[((size_t)s * p.B + b) * p.N + n];
    return v;
  };
  if constexpr (EPI == EPI_SWIGLU) {
    const int n = (c >> 3) * 16 + (c & 7);     // gate row; its up row is 8 further
    reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + c] = from_f<OT>(silu(sum(n)) * sum(n + 8));
  } else if constexpr (EPI == EPI_RESID) {
    reinterpret_cast<float*>(p.out)[(size_t)b * p.ldo + c] += sum(c);
  } else {
    reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + c] = from_f<OT>(sum(c));
  }
}

template <typename TX, typename OT, int NB, int EPI>
static hipError_t gemv_launch(const GemvArgs& p, hipStream_t s) {
  const int splits = EPI == EPI_ARGMAX ? 1 : gemv_splits(p.N, p.K);   // the fused argmax needs whole rows
  const int chunks = p.K / GV_KC;
  const int kc = (chunks + splits - 1) / splits * GV_KC;
  dim3 grid(p.N / (4 * GV_RW), splits);
  if (splits == 1) {
    hipLaunchKernelGGL((gemv_kernel<TX, OT, NB, EPI, true, GV_RW>), grid, dim3(256), 0, s, p, kc);
    return hipGetLastError();
  }
  if (EPI == EPI_ARGMAX || !p.partial) return hipErrorInvalidValue;
  hipLaunchKernelGGL((gemv_kernel<TX, OT, NB, EPI, false, GV_RW>), grid, dim3(256), 0, s, p, kc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.out == nullptr) return e;      // out == null: the caller reduces the partials
  const long n = (long)p.B * (EPI == EPI_SWIGLU ? p.N / 2 : p.N);
  hipLaunchKernelGGL((gemv_reduce<OT, EPI>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, splits);
  return hipGetLastError();
}

template <typename TX, typename OT>
hipError_t gemv(const GemvArgs& p, int epi, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.B > 32 || p.N % 64 || p.K % GV_KC || p.ldx % 8 || p.ldw % 8) return hipErrorInvalidValue;
  if (epi == EPI_ARGMAX && !p.argmax_keys) return hipErrorInvalidValue;
  const bool two = p.B > 16;
#define NOVA_GEMV_CASE(E)                                                             \
  case E: return two ? gemv_launch<TX, OT, 2, E>(p, s) : gemv_launch<TX, OT, 1, E>(p, s);
  switch (epi) {
    NOVA_GEMV_CASE(EPI_STORE)
    NOVA_GEMV_CASE(EPI_RESID)
    NOVA_GEMV_CASE(EPI_SWIGLU)
    NOVA_GEMV_CASE(EPI_ARGMAX)
  }
#undef NOVA_GEMV_CASE
  return hipErrorInvalidValue;
}

template hipError_t gemv<bf16_t, bf16_t>(const GemvArgs&, int, hipStream_t);
template hipError_t gemv<bf16_t, float>(const GemvArgs&, int, hipStream_t);
template hipError_t gemv<float, float>(const GemvArgs&, int, hipStream_t);

}  // namespace nova
