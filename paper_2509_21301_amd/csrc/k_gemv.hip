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
#include "common.hpp"
#include "kernels.hpp"

namespace nova {

constexpr int GV_KC = 256;          // K chunk per pipeline step
constexpr int GV_ROWS = 128;        // weight rows per workgroup (4 waves x 32)

int gemv_splits(int N, int K) {
  const int chunks = K / GV_KC, blocks = N / GV_ROWS;
  if (blocks >= 256) return 1;
  const int want = (256 + blocks - 1) / blocks;
  for (int s = want; s <= chunks; ++s)
    if (chunks % s == 0) return s;
  return chunks;
}

size_t gemv_partial_floats(int B, int N, int K) {
  const int s = gemv_splits(N, K);
  return s > 1 ? (size_t)s * B * N : 0;
}

template <typename TX, typename OT, int NB, int EPI, bool DIRECT>
__global__ void __launch_bounds__(256) gemv_kernel(GemvArgs p, int kc) {
  constexpr bool F32X = sizeof(TX) == 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_base = blockIdx.x * GV_ROWS + wave * 32;
  const int split = blockIdx.y;
  const int k_begin = split * kc, k_end = k_begin + kc;
  const int row = lane & 15, g = lane >> 4;
  // Fragment u of a 256-wide chunk holds k = k0 + 8 * (4u + g) .. +8: the four lanes of a row
  // read 64 adjacent bytes per instruction and two instructions complete each 128-byte line.
  const bf16_t* w0 = p.W + (size_t)(n_base + row) * p.ldw + 8 * g;
  const bf16_t* w1 = w0 + (size_t)16 * p.ldw;
  const TX* X = reinterpret_cast<const TX*>(p.X);

  f32x4 acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load_w = [&](int k0, u32x4 (&wa)[8], u32x4 (&wb)[8]) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      wa[u] = *reinterpret_cast<const u32x4*>(w0 + k0 + 32 * u);
      wb[u] = *reinterpret_cast<const u32x4*>(w1 + k0 + 32 * u);
    }
  };
  auto compute = [&](int k0, const u32x4 (&wa)[8], const u32x4 (&wb)[8]) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int b = j * 16 + row;
      const TX* xr = X + (size_t)b * p.ldx + k0 + 8 * g;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        Frag8 fx, fl;
        if (b < p.B) {
          if constexpr (F32X) {
            float x8[8];
            *reinterpret_cast<float4*>(x8) = *reinterpret_cast<const float4*>(xr + 32 * u);
            *reinterpret_cast<float4*>(x8 + 4) = *reinterpret_cast<const float4*>(xr + 32 * u + 4);
            split8(x8, fx, fl);
          } else {
            fx = *reinterpret_cast<const Frag8*>(xr + 32 * u);
          }
        } else {
          fx = zero_frag();
          if constexpr (F32X) fl = zero_frag();
        }
        acc[0][j] = mfma16(__builtin_bit_cast(Frag8, wa[u]), fx, acc[0][j]);
        acc[1][j] = mfma16(__builtin_bit_cast(Frag8, wb[u]), fx, acc[1][j]);
        if constexpr (F32X) {
          acc[0][j] = mfma16(__builtin_bit_cast(Frag8, wa[u]), fl, acc[0][j]);
          acc[1][j] = mfma16(__builtin_bit_cast(Frag8, wb[u]), fl, acc[1][j]);
        }
      }
    }
  };

  // two chunks per trip: the loads of the next chunk are in flight while this one computes
  u32x4 wa0[8], wb0[8], wa1[8], wb1[8];
  load_w(k_begin, wa0, wb0);
  for (int k0 = k_begin; k0 < k_end; k0 += 2 * GV_KC) {
    const bool has1 = k0 + GV_KC < k_end;
    if (has1) load_w(k0 + GV_KC, wa1, wb1);
    compute(k0, wa0, wb0);
    if (!has1) break;
    if (k0 + 2 * GV_KC < k_end) load_w(k0 + 2 * GV_KC, wa0, wb0);
    compute(k0 + GV_KC, wa1, wb1);
  }

  // lane holds D[n = 4*(lane/16) + r][b = lane%16] of each 16x16 tile
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int b = j * 16 + (lane & 15);
    if (b >= p.B) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int nr = (lane >> 4) * 4 + r;
      if constexpr (!DIRECT) {
        float* part = p.partial + ((size_t)split * p.B + b) * p.N;
        part[n_base + nr] = acc[0][j][r];
        part[n_base + 16 + nr] = acc[1][j][r];
      } else if constexpr (EPI == EPI_SWIGLU) {
        const int oc = (n_base >> 1) + nr;
        reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + oc] = from_f<OT>(silu(acc[0][j][r]) * acc[1][j][r]);
      } else if constexpr (EPI == EPI_RESID) {
        float* o = reinterpret_cast<float*>(p.out) + (size_t)b * p.ldo;
        o[n_base + nr] += acc[0][j][r];
        o[n_base + 16 + nr] += acc[1][j][r];
      } else {
        OT* o = reinterpret_cast<OT*>(p.out) + (size_t)b * p.ldo;
        o[n_base + nr] = from_f<OT>(acc[0][j][r]);
        o[n_base + 16 + nr] = from_f<OT>(acc[1][j][r]);
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
    for (int s = 0; s < splits; ++s) v += p.partial[((size_t)s * p.B + b) * p.N + n];
    return v;
  };
  if constexpr (EPI == EPI_SWIGLU) {
    const int n = (c >> 4) * 32 + (c & 15);
    reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + c] = from_f<OT>(silu(sum(n)) * sum(n + 16));
  } else if constexpr (EPI == EPI_RESID) {
    reinterpret_cast<float*>(p.out)[(size_t)b * p.ldo + c] += sum(c);
  } else {
    reinterpret_cast<OT*>(p.out)[(size_t)b * p.ldo + c] = from_f<OT>(sum(c));
  }
}

template <typename TX, typename OT, int NB, int EPI>
static hipError_t gemv_launch(const GemvArgs& p, hipStream_t s) {
  const int splits = gemv_splits(p.N, p.K);
  const int kc = p.K / splits;
  dim3 grid(p.N / GV_ROWS, splits);
  if (splits == 1) {
    hipLaunchKernelGGL((gemv_kernel<TX, OT, NB, EPI, true>), grid, dim3(256), 0, s, p, kc);
    return hipGetLastError();
  }
  if (!p.partial) return hipErrorInvalidValue;
  hipLaunchKernelGGL((gemv_kernel<TX, OT, NB, EPI, false>), grid, dim3(256), 0, s, p, kc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long n = (long)p.B * (EPI == EPI_SWIGLU ? p.N / 2 : p.N);
  hipLaunchKernelGGL((gemv_reduce<OT, EPI>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, splits);
  return hipGetLastError();
}

template <typename TX, typename OT>
hipError_t gemv(const GemvArgs& p, int epi, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.B > 32 || p.N % GV_ROWS || p.K % GV_KC || p.ldx % 8 || p.ldw % 8) return hipErrorInvalidValue;
  const bool two = p.B > 16;
#define NOVA_GEMV_CASE(E)                                                             \
  case E: return two ? gemv_launch<TX, OT, 2, E>(p, s) : gemv_launch<TX, OT, 1, E>(p, s);
  switch (epi) {
    NOVA_GEMV_CASE(EPI_STORE)
    NOVA_GEMV_CASE(EPI_RESID)
    NOVA_GEMV_CASE(EPI_SWIGLU)
  }
#undef NOVA_GEMV_CASE
  return hipErrorInvalidValue;
}

template hipError_t gemv<bf16_t, bf16_t>(const GemvArgs&, int, hipStream_t);
template hipError_t gemv<bf16_t, float>(const GemvArgs&, int, hipStream_t);
template hipError_t gemv<float, float>(const GemvArgs&, int, hipStream_t);

}  // namespace nova
