// Dense GEMM for the encode and prefill linears: C[M,N] = A[M,K] . W[N,K]^T with a fused epilogue.
//
// These are the QKV, output-projection, MLP up/gate and down linears that dominate vision encode
// and prefill time (the paper's Table 3 and Sec. 3.2.1).  Design for gfx950:
//  * bf16 MFMA 16x16x32 (fp32 accumulate); four waves per workgroup, each owning a WM x WN tile;
//  * A and W tiles staged through LDS with a 16-byte row pad (conflict-free ds_read_b128),
//    double-buffered so the global loads of tile k+1 overlap the MFMAs of tile k;
//  * tile order remapped so that each XCD (which owns one L2) works on a contiguous block of
//    output tiles: the dispatcher deals workgroups to the 8 XCDs round-robin;
//  * fp32 activations (tiny-stack exact mode) are split into bf16 hi + lo parts, two MFMAs each,
//    since weights are exactly bf16.
// Requirements (checked by the host): N % BN == 0, K % 64 == 0, 16-byte aligned rows.
#include "common.hpp"
#include "kernels.hpp"

namespace nova {

constexpr int BK = 64;
constexpr int PAD = 8;             // bf16 elements of row padding in LDS
constexpr int LDK = BK + PAD;      // LDS row pitch (elements)

template <typename TA, typename OT, int EPI, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64) gemm_kernel(GemmArgs p) {
  constexpr bool F32A = sizeof(TA) == 4;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int WAVES_N = BN / WN;
  constexpr int NT = (BM / WM) * (BN / WN) * 64;     // threads per workgroup
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* As = reinterpret_cast<bf16_t*>(smem);                 // [2][BM][LDK] (x2 for hi/lo)
  constexpr int A_ELEMS = BM * LDK * (F32A ? 2 : 1);
  bf16_t* Bs = As + 2 * A_ELEMS;                                 // [2][BN][LDK]
  constexpr int B_ELEMS = BN * LDK;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  // ---- tile index: XCD-contiguous, then grouped along M for L2 reuse of W
  const int nm = (p.M + BM - 1) / BM, nn = p.N / BN;
  const int total = nm * nn;
  int id = blockIdx.x;
  if ((total & 7) == 0) id = (id & 7) * (total >> 3) + (id >> 3);
  constexpr int G = 8;
  const int group = id / (G * nn);
  const int first_m = group * G;
  const int gsize = min(nm - first_m, G);
  const int within = id % (G * nn);
  const int tile_m = first_m + within % gsize;
  const int tile_n = within / gsize;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  // ---- global -> register staging
  constexpr int A_CHUNK = F32A ? 4 : 8;                 // elements per 16-byte chunk
  constexpr int A_CPR = BK / A_CHUNK;                   // chunks per row
  constexpr int A_ITERS = BM * A_CPR / NT;
  constexpr int B_ITERS = BN * (BK / 8) / NT;
  static_assert(A_ITERS * NT == BM * A_CPR && B_ITERS * NT == BN * (BK / 8), "tile/thread mismatch");
  u32x4 ra[A_ITERS], rb[B_ITERS];
  const TA* Ag = reinterpret_cast<const TA*>(p.A);

  auto load_global = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_ITERS; ++i) {
      int c = tid + i * NT, row = c / A_CPR, col = (c % A_CPR) * A_CHUNK;
      int m = m0 + row;
      if (m < p.M) ra[i] = *reinterpret_cast<const u32x4*>(Ag + (size_t)m * p.lda + k0 + col);
      else ra[i] = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < B_ITERS; ++i) {
      int c = tid + i * NT, row = c / (BK / 8), col = (c % (BK / 8)) * 8;
      rb[i] = *reinterpret_cast<const u32x4*>(p.W + (size_t)(n0 + row) * p.ldw + k0 + col);
    }
  };
  auto store_lds = [&](int buf) {
    bf16_t* a = As + buf * A_ELEMS;
    bf16_t* b = Bs + buf * B_ELEMS;
#pragma unroll
    for (int i = 0; i < A_ITERS; ++i) {
      int c = tid + i * NT, row = c / A_CPR, col = (c % A_CPR) * A_CHUNK;
      if constexpr (F32A) {
        float x[4] = {__uint_as_float(ra[i][0]), __uint_as_float(ra[i][1]), __uint_as_float(ra[i][2]),
                      __uint_as_float(ra[i][3])};
        bf16_t h[4];
        float l[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) { h[j] = f2bf(x[j]); l[j] = x[j] - bf2f(h[j]); }
        uint2 hv = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
        uint2 lv = make_uint2(pack2(l[0], l[1]), pack2(l[2], l[3]));
        *reinterpret_cast<uint2*>(a + row * LDK + col) = hv;
        *reinterpret_cast<uint2*>(a + BM * LDK + row * LDK + col) = lv;
      } else {
        *reinterpret_cast<u32x4*>(a + row * LDK + col) = ra[i];
      }
    }
#pragma unroll
    for (int i = 0; i < B_ITERS; ++i) {
      int c = tid + i * NT, row = c / (BK / 8), col = (c % (BK / 8)) * 8;
      *reinterpret_cast<u32x4*>(b + row * LDK + col) = rb[i];
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = p.K / BK;
  load_global(0);
  store_lds(0);
  __syncthreads();

  const int fr = lane & 15, fk = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_global((kt + 1) * BK);
    const bf16_t* a = As + cur * A_ELEMS;
    const bf16_t* b = Bs + cur * B_ELEMS;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      Frag8 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *reinterpret_cast<const Frag8*>(a + (wm * WM + i * 16 + fr) * LDK + kk + fk);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *reinterpret_cast<const Frag8*>(b + (wn * WN + j * 16 + fr) * LDK + kk + fk);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(fa[i], fb[j], acc[i][j]);
      if constexpr (F32A) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
          fa[i] = *reinterpret_cast<const Frag8*>(a + BM * LDK + (wm * WM + i * 16 + fr) * LDK + kk + fk);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(fa[i], fb[j], acc[i][j]);
      }
    }
    if (kt + 1 < nk) store_lds(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds rows 4*(lane/16)+r, column lane%16 of each 16x16 tile
  const int er = (lane >> 4) * 4, ec = lane & 15;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * WM + i * 16 + er + r;
      if (m >= p.M) continue;
      if constexpr (EPI == EPI_SWIGLU) {
        // W rows interleaved in blocks of 8: columns 0-7 of each 16-wide tile are gate outputs,
        // 8-15 the matching up outputs, held by lanes 8 apart
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const float g = acc[i][j][r], u = __shfl_xor(acc[i][j][r], 8, 64);
          if (ec < 8) {
            const int oc = ((n0 + wn * WN + j * 16) >> 1) + ec;
            reinterpret_cast<OT*>(p.out)[(size_t)m * p.ldo + oc] = from_f<OT>(silu(g) * u);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int n = n0 + wn * WN + j * 16 + ec;
          float v = acc[i][j][r];
          if (p.bias) v += bf2f(p.bias[n]);
          if constexpr (EPI == EPI_STORE) {
            reinterpret_cast<OT*>(p.out)[(size_t)m * p.ldo + n] = from_f<OT>(v);
          } else if constexpr (EPI == EPI_GELU) {
            reinterpret_cast<OT*>(p.out)[(size_t)m * p.ldo + n] = from_f<OT>(gelu_erf(v));
          } else if constexpr (EPI == EPI_RESID) {
            float* o = reinterpret_cast<float*>(p.out) + (size_t)m * p.ldo + n;
            *o = *o + v;
          } else if constexpr (EPI == EPI_POS) {
            float* o = reinterpret_cast<float*>(p.out) + (size_t)m * p.ldo + n;
            *o = v + bf2f(p.pos[(size_t)(m % p.pos_rows) * p.N + n]);
          }
        }
      }
    }
  }
}

template <typename TA, typename OT, int EPI, int BM, int BN, int WM, int WN>
static hipError_t launch_tile(const GemmArgs& p, hipStream_t s) {
  constexpr bool F32A = sizeof(TA) == 4;
  const size_t lds = (size_t)2 * (BM * LDK * (F32A ? 2 : 1) + BN * LDK) * sizeof(bf16_t);
  auto kern = gemm_kernel<TA, OT, EPI, BM, BN, WM, WN>;
  static bool attr_set = false;   // benign race: idempotent attribute
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int nm = (p.M + BM - 1) / BM, nn = p.N / BN;
  hipLaunchKernelGGL(kern, dim3(nm * nn), dim3((BM / WM) * (BN / WN) * 64), lds, s, p);
  return hipGetLastError();
}

template <typename TA, typename OT, int EPI>
static hipError_t launch_epi(const GemmArgs& p, hipStream_t s) {
  // 256x256 tiles with 8 waves (two per SIMD, each 64x128) when N is wide and there are at least
  // two tiles per CU; otherwise 128x128 tiles with 4 waves (two workgroups per CU).
  if constexpr (sizeof(TA) == 2) {
    const long tiles = (long)((p.M + 255) / 256) * (p.N / 256);
    if (p.N % 256 == 0 && p.N >= 3072 && tiles >= 512) return launch_tile<TA, OT, EPI, 256, 256, 64, 128>(p, s);
  }
  return launch_tile<TA, OT, EPI, 128, 128, 64, 64>(p, s);
}

template <typename TA, typename OT>
hipError_t gemm(const GemmArgs& p, int epi, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (p.N % 128 || p.K % BK || p.lda % 8 || p.ldw % 8) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE: return launch_epi<TA, OT, EPI_STORE>(p, s);
    case EPI_GELU: return launch_epi<TA, OT, EPI_GELU>(p, s);
    case EPI_RESID: return launch_epi<TA, OT, EPI_RESID>(p, s);
    case EPI_POS: return launch_epi<TA, OT, EPI_POS>(p, s);
    case EPI_SWIGLU: return launch_epi<TA, OT, EPI_SWIGLU>(p, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t gemm<bf16_t, bf16_t>(const GemmArgs&, int, hipStream_t);
template hipError_t gemm<float, float>(const GemmArgs&, int, hipStream_t);

}  // namespace nova
