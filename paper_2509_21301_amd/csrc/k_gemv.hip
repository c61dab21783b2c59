// Thin GEMM for the decode linears and the LM head: Y[B,N] = X[B,K] W[N,K]^T, B <= 32.
//
// Decode is bound by streaming the weights from HBM (the paper's Table 3 decode row and
// Sec. 3.2.1).  Each wave streams 32 weight rows with 16-byte loads, 128 contiguous bytes per
// lane per 256-wide K chunk (16 loads in flight per lane), and feeds them to MFMA 16x16x32 as
// the A operand with the batch as the 16-wide B operand (a second MFMA covers rows 16..31 of
// the batch).  X chunks are staged in LDS once per workgroup.  When N alone gives too few
// workgroups, K is split and a small second pass reduces the fp32 partials and applies the
// epilogue; otherwise the epilogue is applied directly.
// The k index of an MFMA fragment only has to agree between its A and B operands, so each
// lane can read 128 contiguous bytes of its row and use them as eight consecutive fragments.
#include "common.hpp"
#include "kernels.hpp"

namespace nova {

constexpr int GV_KC = 256;          // K chunk staged per iteration
constexpr int GV_XP = GV_KC + 8;    // LDS row pitch of the X chunk (bf16 elements)
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
  __shared__ __align__(16) bf16_t xs[(F32X ? 2 : 1) * 32 * GV_XP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_base = blockIdx.x * GV_ROWS + wave * 32;
  const int split = blockIdx.y;
  const int k_begin = split * kc;
  const int row = lane & 15, g = lane >> 4;
  const bf16_t* w0 = p.W + (size_t)(n_base + row) * p.ldw;
  const bf16_t* w1 = w0 + (size_t)16 * p.ldw;
  const TX* X = reinterpret_cast<const TX*>(p.X);

  f32x4 acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = k_begin; k0 < k_begin + kc; k0 += GV_KC) {
    // weight fragments for this chunk: 128 contiguous bytes of each of the lane's two rows
    u32x4 wa[8], wb[8];
    const u32x4* pa = reinterpret_cast<const u32x4*>(w0 + k0 + g * 64);
    const u32x4* pb = reinterpret_cast<const u32x4*>(w1 + k0 + g * 64);
#pragma unroll
    for (int u = 0; u < 8; ++u) { wa[u] = __builtin_nontemporal_load(pa + u); wb[u] = __builtin_nontemporal_load(pb + u); }
    // stage X[0..31][k0..k0+255] (rows >= B are zero)
    __syncthreads();
    if constexpr (F32X) {
      for (int c = tid; c < 32 * GV_KC / 4; c += 256) {
        const int b = c / (GV_KC / 4), col = (c % (GV_KC / 4)) * 4;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if (b < p.B) {
          float4 t = *reinterpret_cast<const float4*>(X + (size_t)b * p.ldx + k0 + col);
          v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
        }
        bf16_t h[4];
        float l[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) { h[j] = f2bf(v[j]); l[j] = v[j] - bf2f(h[j]); }
        *reinterpret_cast<uint2*>(xs + b * GV_XP + col) =
            make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
        *reinterpret_cast<uint2*>(xs + 32 * GV_XP + b * GV_XP + col) = make_uint2(pack2(l[0], l[1]), pack2(l[2], l[3]));
      }
    } else {
      for (int c = tid; c < 32 * GV_KC / 8; c += 256) {
        const int b = c / (GV_KC / 8), col = (c % (GV_KC / 8)) * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (b < p.B) v = *reinterpret_cast<const uint4*>(X + (size_t)b * p.ldx + k0 + col);
        *reinterpret_cast<uint4*>(xs + b * GV_XP + col) = v;
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int kk = g * 64 + u * 8;
      Frag8 fa = __builtin_bit_cast(Frag8, wa[u]);
      Frag8 fb = __builtin_bit_cast(Frag8, wb[u]);
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        Frag8 fx = *reinterpret_cast<const Frag8*>(xs + (j * 16 + row) * GV_XP + kk);
        acc[0][j] = mfma16(fa, fx, acc[0][j]);
        acc[1][j] = mfma16(fb, fx, acc[1][j]);
        if constexpr (F32X) {
          Frag8 fl = *reinterpret_cast<const Frag8*>(xs + 32 * GV_XP + (j * 16 + row) * GV_XP + kk);
          acc[0][j] = mfma16(fa, fl, acc[0][j]);
          acc[1][j] = mfma16(fb, fl, acc[1][j]);
        }
      }
    }
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
