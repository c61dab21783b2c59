// Dense GEMM for the encode and prefill linears: C[M,N] = A[M,K] . W[N,K]^T with a fused epilogue.
//
// These are the QKV, output-projection, MLP up/gate and down linears that dominate vision encode
// and prefill time (the paper's Table 3 and Sec. 3.2.1).  Design for gfx950:
//  * bf16 MFMA 16x16x32 (fp32 accumulate); 4 or 8 waves per workgroup, each owning a WM x WN tile;
//  * bf16 activations: A and W tiles go global -> LDS by 16-byte LDS-DMA loads in an XOR-swizzled
//    layout (conflict-free fragment reads), two stages, the DMA of step k+1 in flight during the
//    MFMAs of step k;
//  * fp32 activations (tiny-stack exact mode): tiles staged through registers (split into bf16
//    hi + lo parts, two MFMAs each, since weights are exactly bf16) into a padded LDS layout;
//  * tile order remapped so that each XCD (which owns one L2) works on a contiguous block of
//    output tiles: the dispatcher deals workgroups to the 8 XCDs round-robin;
//  * the epilogue (bias, GELU, SwiGLU, residual or position add) runs through LDS so that every
//    global access covers whole cache lines.
// Requirements (checked by the host): N % 128 == 0, K % 64 == 0, 16-byte aligned rows, ldo % 4 == 0.
#include "common.hpp"
#include "kernels.hpp"

namespace nova {

// The dispatcher deals workgroup b of a launch to XCD b % 8.  Renumbered so that each XCD takes
// one contiguous range of the n tile ids (the first n % 8 XCDs one more than the others), the
// tiles resident on an XCD at a time are neighbours and share A and W panels in its L2, whatever
// n is (with an 8-way round-robin of plain ids, no two neighbouring tiles share an L2).
__device__ __forceinline__ int xcd_contiguous(int b, int n) {
  const int q = n >> 3, r = n & 7, x = b & 7, j = b >> 3;
  return x < r ? x * (q + 1) + j : r * (q + 1) + (x - r) * q + j;
}

constexpr int BK = 64;
constexpr int PAD = 8;             // bf16 elements of row padding in LDS
constexpr int LDK = BK + PAD;      // LDS row pitch (elements)

// Four consecutive outputs: one 16-byte (fp32) or 8-byte (bf16) store.
template <typename OT>
__device__ __forceinline__ void store4(OT* dst, const float v[4]) {
  if constexpr (sizeof(OT) == 4) {
    *reinterpret_cast<float4*>(dst) = float4{v[0], v[1], v[2], v[3]};
  } else {
    *reinterpret_cast<uint2*>(dst) = make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
  }
}

// Epilogue, through LDS (free after the main loop's last barrier): each wave stages one 16-row
// block of its WM x WN tile at a time in a private fp32 scratch, then reads it back along rows so
// that every global access covers whole cache lines (the MFMA layout gives a lane one column
// of 4 rows).  row0/col0: the wave tile's first output row and column.
template <typename OT, int EPI, int WM, int WN>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& p, const f32x4 (&acc)[WM / 16][WN / 16], float* smem,
                                              int wave, int lane, int row0, int col0) {
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int SP = WN + 4;                         // scratch pitch: the writes of rows 4 apart
  constexpr bool SW = EPI == EPI_SWIGLU;
  constexpr int LPR = SW ? WN / 8 : WN / 4;          // lanes per scratch row
  constexpr int RPI = 64 / LPR, NP = 16 / RPI;       // rows per pass, passes per block
  float* sc = smem + wave * 16 * SP;                 // land 16 banks apart
  const int er = (lane >> 4) * 4, ec = lane & 15;
  const int q = lane % LPR, prow = lane / LPR;
  // this lane's columns are the same in every pass: 4 consecutive ones, or for SwiGLU (W rows
  // interleaved in blocks of 8: of each 16 columns, 0-7 gate and 8-15 the matching up rows)
  // 4 gate columns and the 4 up columns 8 further, giving 4 outputs
  if constexpr (EPI == EPI_STORE) {
    if (p.vt != nullptr && col0 >= p.v_col0) {
      // V columns of a fused QKV projection go to V^T.  bf16: 64 columns at a time are staged in
      // the wave's LDS scratch transposed ([column][WM tokens + 8], each lane writing its 4
      // consecutive tokens of one column as 8 bytes), then every V^T row segment of WM tokens
      // leaves as whole 16-byte pieces.  fp32 (exact mode): one 16-byte store per lane and tile.
      const int er = (lane >> 4) * 4, ec = lane & 15;
      const int heads = (p.N - p.v_col0) / p.vt_hd;
      OT* vt = reinterpret_cast<OT*>(p.vt);
      if constexpr (sizeof(OT) == 2) {
        constexpr int TP = WM + 8;                 // bf16 pitch of a staged column
        constexpr int TN2 = TN < 4 ? TN : 4;       // 16-column blocks per pass
        constexpr int CH = WM / 8;                 // 16-byte pieces per staged column
        bf16_t* tl = reinterpret_cast<bf16_t*>(smem) + wave * (TN2 * 16) * TP;
#pragma unroll
        for (int jh = 0; jh < TN; jh += TN2) {
#pragma unroll
          for (int j = 0; j < TN2; ++j) {
            const int n = col0 + (jh + j) * 16 + ec;
            const float bv = p.bias ? bf2f(p.bias[n]) : 0.f;
#pragma unroll
            for (int i = 0; i < TM; ++i)
              *reinterpret_cast<uint2*>(tl + (j * 16 + ec) * TP + i * 16 + er) =
                  make_uint2(pack2(acc[i][jh + j][0] + bv, acc[i][jh + j][1] + bv),
                             pack2(acc[i][jh + j][2] + bv, acc[i][jh + j][3] + bv));
          }
          asm volatile("" ::: "memory");     // a wave's LDS operations execute in order
#pragma unroll
          for (int q = lane; q < TN2 * 16 * CH; q += 64) {
            const int cc = q / CH, m = row0 + (q % CH) * 8;     // 8 tokens, never across images
            if (m < p.M) {
              const int mg = m + p.vt_row0, b = mg / p.vt_tokens, t = mg - b * p.vt_tokens;
              const int c = col0 + jh * 16 + cc - p.v_col0, h = c / p.vt_hd, d = c - h * p.vt_hd;
              *reinterpret_cast<u32x4*>(vt + ((size_t)(b * heads + h) * p.vt_hd + d) * p.vt_pad + t) =
                  *reinterpret_cast<const u32x4*>(tl + cc * TP + (q % CH) * 8);
            }
          }
          asm volatile("" ::: "memory");
        }
      } else {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int m = row0 + i * 16 + er;
          if (m >= p.M) continue;
          const int mg = m + p.vt_row0, b = mg / p.vt_tokens, t = mg - b * p.vt_tokens;
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int n = col0 + j * 16 + ec, c = n - p.v_col0;
            const int h = c / p.vt_hd, d = c - h * p.vt_hd;
            const float bv = p.bias ? bf2f(p.bias[n]) : 0.f;
            const float o[4] = {acc[i][j][0] + bv, acc[i][j][1] + bv, acc[i][j][2] + bv, acc[i][j][3] + bv};
            store4<OT>(vt + ((size_t)(b * heads + h) * p.vt_hd + d) * p.vt_pad + t, o);
          }
        }
      }
      return;
    }
  }
  const int c = SW ? (q >> 1) * 16 + (q & 1) * 4 : q * 4;
  const int n = col0 + c;
  const int nout = SW ? (col0 >> 1) + (q >> 1) * 8 + (q & 1) * 4 : n;
  float bias[4] = {0.f, 0.f, 0.f, 0.f};
  if constexpr (!SW) {
    if (p.bias) {
      const uint2 bb = *reinterpret_cast<const uint2*>(p.bias + n);
      bias[0] = bf2f((bf16_t)(bb.x & 0xffff)); bias[1] = bf2f((bf16_t)(bb.x >> 16));
      bias[2] = bf2f((bf16_t)(bb.y & 0xffff)); bias[3] = bf2f((bf16_t)(bb.y >> 16));
    }
  }
  // residual / position rows of block i (rows past M clamped): the next block's are loaded
  // while this block goes through the scratch, so one load latency is exposed per tile
  constexpr bool XIN = EPI == EPI_RESID || EPI == EPI_POS;
  auto load_x = [&](int i, float4 (&x)[NP]) {
#pragma unroll
    for (int t = 0; t < NP; ++t) {
      const int m = min(row0 + i * 16 + t * RPI + prow, p.M - 1);
      if constexpr (EPI == EPI_RESID) {
        x[t] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p.out) + (size_t)m * p.ldo + n);
      } else {
        const uint2 pp = *reinterpret_cast<const uint2*>(p.pos + (size_t)(m % p.pos_rows) * p.N + n);
        x[t] = float4{bf2f((bf16_t)(pp.x & 0xffff)), bf2f((bf16_t)(pp.x >> 16)),
                      bf2f((bf16_t)(pp.y & 0xffff)), bf2f((bf16_t)(pp.y >> 16))};
      }
    }
  };
  float4 xb[2][XIN ? NP : 1];
  if constexpr (XIN) load_x(0, xb[0]);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    if constexpr (XIN) {
      if (i + 1 < TM) load_x(i + 1, xb[(i + 1) & 1]);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) sc[(er + r) * SP + j * 16 + ec] = acc[i][j][r];
    // a wave's LDS operations execute in order; keep the compiler from reordering them
    asm volatile("" ::: "memory");
    float4 v[NP], u[NP];
#pragma unroll
    for (int t = 0; t < NP; ++t) {
      const int row = t * RPI + prow;
      v[t] = *reinterpret_cast<const float4*>(sc + row * SP + c);
      if constexpr (SW) u[t] = *reinterpret_cast<const float4*>(sc + row * SP + c + 8);
    }
    asm volatile("" ::: "memory");
    const float4* x = xb[i & 1];
#pragma unroll
    for (int t = 0; t < NP; ++t) {
      const int m = row0 + i * 16 + t * RPI + prow;
      if (m >= p.M) continue;
      float o[4] = {v[t].x + bias[0], v[t].y + bias[1], v[t].z + bias[2], v[t].w + bias[3]};
      if constexpr (SW) {
        o[0] = silu(v[t].x) * u[t].x; o[1] = silu(v[t].y) * u[t].y;
        o[2] = silu(v[t].z) * u[t].z; o[3] = silu(v[t].w) * u[t].w;
        store4<OT>(reinterpret_cast<OT*>(p.out) + (size_t)m * p.ldo + nout, o);
      } else if constexpr (EPI == EPI_STORE) {
        store4<OT>(reinterpret_cast<OT*>(p.out) + (size_t)m * p.ldo + n, o);
      } else if constexpr (EPI == EPI_GELU) {
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = gelu_erf(o[e]);
        store4<OT>(reinterpret_cast<OT*>(p.out) + (size_t)m * p.ldo + n, o);
      } else {   // RESID, POS: fp32 out
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(p.out) + (size_t)m * p.ldo + n) =
            float4{o[0] + x[t].x, o[1] + x[t].y, o[2] + x[t].z, o[3] + x[t].w};
      }
    }
  }
}

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
  const int id = xcd_contiguous(blockIdx.x, gridDim.x);
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

  gemm_epilogue<OT, EPI, WM, WN>(p, acc, reinterpret_cast<float*>(smem), wave, lane, m0 + wm * WM, n0 + wn * WN);
}

// bf16 activations: both tiles go global -> LDS directly (16-byte LDS-DMA loads, no register
// staging), two LDS stages, one barrier per 64-wide K step.  A DMA instruction fills 1 KB of LDS
// in lane order, i.e. 8 rows x 128 bytes; each lane picks the k piece that belongs in its slot,
// so the tile is stored with piece p of row r at slot p ^ ((r / 2) % 8), which makes the
// 16-row MFMA fragment reads conflict-free.  Rows past M are clamped to M - 1 (they feed only
// output rows that are never stored), so every load is unconditional.
// One 16-byte-per-lane LDS-DMA load: lane l's 16 bytes from g land at l_base + 16 * l.
__device__ __forceinline__ void lds_dma16(const bf16_t* g, bf16_t* l_base) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)l_base, 16, 0, 0);
}

// The same 16-byte LDS-DMA load written as inline assembly, to the LDS byte address lds_addr
// (wave-uniform, passed in M0).  The compiler does not track it: a fragment read that follows it
// in program order is not made to wait for it, so the caller orders DMA and reads itself with
// s_waitcnt and barriers.
__device__ __forceinline__ void lds_dma16_untracked(const bf16_t* g, uint32_t lds_addr) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"{m0}"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(g)
               : "memory");
}
__device__ __forceinline__ uint32_t lds_addr_of(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

template <typename OT, int EPI, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64) gemm_dma_kernel(GemmArgs p) {
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int WAVES_N = BN / WN;
  constexpr int NW = (BM / WM) * (BN / WN);
  constexpr int STAGE = (BM + BN) * BK;              // bf16 per stage
  constexpr int IA = BM / 8 / NW, IB = BN / 8 / NW;  // DMA instructions per wave per stage
  static_assert(IA * NW * 8 == BM && IB * NW * 8 == BN, "tile rows must split into 8-row DMA groups");
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  const int nm = (p.M + BM - 1) / BM, nn = p.N / BN;
  const int total = nm * nn;
  // split K: workgroup blockIdx.x / total takes K slice number that many, writing fp32 partials
  const int idg = xcd_contiguous(blockIdx.x, gridDim.x);
  const int ks = p.kslice ? idg / total : 0;
  const int id = idg - ks * total;
  // groups of G M-tiles sweep the N tiles together (an XCD's ~32 resident tiles then share a few
  // A and W panels in its L2): 256-row tiles in groups of 4 when there are many row tiles (the
  // XCD's A panels stay in its L2 while the group sweeps N: encode GEMM family 53.1 -> 50.7 ms
  // per pass against groups of 16, one-image encode 14.04 -> 13.87 ms), of 16 (all of them) when
  // there are at most 16 (the 1500-token prefill: 20.30 -> 20.03 ms against groups of 4); 8 for
  // 128-row tiles
  const int G = BM >= 256 ? (nm <= 16 ? 16 : 4) : 8;
  const int group = id / (G * nn);
  const int first_m = group * G;
  const int gsize = min(nm - first_m, G);
  const int within = id % (G * nn);
  const int tile_m = first_m + within % gsize;
  const int tile_n = within / gsize;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  // DMA sources: lane l of a group fills row 8q + l/8, slot l%8 with piece (l%8) ^ ((row/2)%8)
  const size_t k_off = (size_t)ks * p.kslice;
  const bf16_t* A = reinterpret_cast<const bf16_t*>(p.A) + k_off;
  const int lrow = lane >> 3, lslot = lane & 7;
  const bf16_t* asrc[IA];
  const bf16_t* bsrc[IB];
#pragma unroll
  for (int t = 0; t < IA; ++t) {
    const int r = (wave * IA + t) * 8 + lrow;
    asrc[t] = A + (size_t)min(m0 + r, p.M - 1) * p.lda + 8 * (lslot ^ ((r >> 1) & 7));
  }
#pragma unroll
  for (int t = 0; t < IB; ++t) {
    const int r = (wave * IB + t) * 8 + lrow;
    bsrc[t] = p.W + k_off + (size_t)(n0 + r) * p.ldw + 8 * (lslot ^ ((r >> 1) & 7));
  }
  auto dma = [&](int kt, int stage) {
    bf16_t* a = lds + stage * STAGE;
    bf16_t* b = a + BM * BK;
    const int k0 = kt * BK;
#pragma unroll
    for (int t = 0; t < IA; ++t)
      lds_dma16(asrc[t] + k0, a + (wave * IA + t) * 8 * BK);
#pragma unroll
    for (int t = 0; t < IB; ++t)
      lds_dma16(bsrc[t] + k0, b + (wave * IB + t) * 8 * BK);
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // fragment reads: row fr of a 16-row block, k piece 4s + fk of the 64-wide step; the block
  // base is a multiple of 16 rows, so the swizzle depends on fr only
  const int fr = lane & 15, fk = lane >> 4;
  const int sw = (fr >> 1) & 7;
  const int off0 = fr * BK + 8 * (fk ^ sw);          // elements, sub-step 0
  const int off1 = fr * BK + 8 * ((fk + 4) ^ sw);    // sub-step 1
  // K slices are kslice long except the last, which takes what remains
  const int nk = (p.kslice ? min(p.kslice, p.K - (int)k_off) : p.K) / BK;
  if constexpr (BM == 256 && BN == 256 && WM == 64 && WN == 128) {
    // 256x256 tiles (the same schedule measured slower for the 4-wave 128x128 tiles, whose
    // halves have too few MFMAs to cover the reads).  Each 64-wide K step is two halves of TM x TN
    // MFMAs per wave.  A wave reads the fragments
    // of the next half and issues its share of the next stage's DMA in groups spread between the
    // MFMA rows of the current half, so LDS reads, DMA and MFMAs overlap instead of running as
    // phases; one wait and barrier per step sits between the two halves.  The DMA is the
    // untracked form (the compiler would otherwise make each fragment read wait for every DMA in
    // flight); stage s+1 lands while stage s is multiplied.
    constexpr int NF = TM + TN, RPG = NF / TM;     // fragments per half, fragment reads per MFMA row
    static_assert(RPG * TM == NF, "fragment reads must split evenly over the MFMA rows");
    const uint32_t lbase = lds_addr_of(lds);
    uint32_t dst[IA + IB];
    const bf16_t* src[IA + IB];
#pragma unroll
    for (int t = 0; t < IA; ++t) {
      src[t] = asrc[t];
      dst[t] = (uint32_t)((wave * IA + t) * 8 * BK) * 2u;
    }
#pragma unroll
    for (int t = 0; t < IB; ++t) {
      src[IA + t] = bsrc[t];
      dst[IA + t] = (uint32_t)(BM * BK + (wave * IB + t) * 8 * BK) * 2u;
    }
    Frag8 xa[TM], xb[TN], ya[TM], yb[TN];
    // fragment idx (0..NF-1) of a half: A rows 0..TM-1, then B columns 0..TN-1
    auto rd = [&](int stage, int off, int idx, Frag8 (&fa)[TM], Frag8 (&fb)[TN]) {
      const bf16_t* base = lds + stage * STAGE;
      if (idx < TM) fa[idx] = *reinterpret_cast<const Frag8*>(base + (wm * WM + idx * 16) * BK + off);
      else fb[idx - TM] = *reinterpret_cast<const Frag8*>(base + BM * BK + (wn * WN + (idx - TM) * 16) * BK + off);
    };
    // MFMA row i of (ca, cb) for i = 0..TM-1, each preceded by RPG fragment reads of the next half
    // (stage rstage, offset roff) and 2 DMA instructions of K step dkt (if dkt >= 0) into dstage
    auto half = [&](const Frag8 (&ca)[TM], const Frag8 (&cb)[TN], int rstage, int roff, Frag8 (&na)[TM],
                    Frag8 (&nb)[TN], bool do_read, int dkt, int dstage) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        __builtin_amdgcn_sched_barrier(0);
        if (dkt >= 0) {
#pragma unroll
          for (int t = 0; t < 2; ++t)
            lds_dma16_untracked(src[2 * i + t] + dkt * BK, lbase + (uint32_t)(dstage * STAGE) * 2u + dst[2 * i + t]);
        }
        if (do_read) {
#pragma unroll
          for (int r = 0; r < RPG; ++r) rd(rstage, roff, RPG * i + r, na, nb);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(ca[i], cb[j], acc[i][j]);
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    // prologue: stages 0 and 1 in flight, wait for stage 0, read the first half of stage 0
#pragma unroll
    for (int t = 0; t < IA + IB; ++t) lds_dma16_untracked(src[t], lbase + dst[t]);
    if (nk > 1) {
#pragma unroll
      for (int t = 0; t < IA + IB; ++t) lds_dma16_untracked(src[t] + BK, lbase + (uint32_t)STAGE * 2u + dst[t]);
      __builtin_amdgcn_s_waitcnt(0x0F70 | (IA + IB));   // vmcnt(8): stage 0 landed, stage 1 may fly
    } else {
      __builtin_amdgcn_s_waitcnt(0);
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < NF; ++r) rd(0, off0, r, xa, xb);
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      half(xa, xb, cur, off1, ya, yb, true, -1, 0);          // first half; read the second half
      __builtin_amdgcn_s_waitcnt(0);                          // own DMA of stage kt+1 and own reads done
      __syncthreads();                                        // everyone's: stage kt+1 visible, buffer cur free
      half(ya, yb, cur ^ 1, off0, xa, xb, kt + 1 < nk, kt + 2 < nk ? kt + 2 : -1, cur);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();                                          // the epilogue reuses the stage buffers
  } else {
  dma(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const bf16_t* a = lds + (kt & 1) * STAGE + wm * WM * BK;
    const bf16_t* b = lds + (kt & 1) * STAGE + BM * BK + wn * WN * BK;
    Frag8 fa[2][TM], fb[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      fa[0][i] = *reinterpret_cast<const Frag8*>(a + i * 16 * BK + off0);
      fa[1][i] = *reinterpret_cast<const Frag8*>(a + i * 16 * BK + off1);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      fb[0][j] = *reinterpret_cast<const Frag8*>(b + j * 16 * BK + off0);
      fb[1][j] = *reinterpret_cast<const Frag8*>(b + j * 16 * BK + off1);
    }
    // the next stage's DMA is issued after this stage's reads, so that no read has to wait for it
    __builtin_amdgcn_sched_barrier(0);
    if (kt + 1 < nk) dma(kt + 1, (kt + 1) & 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(fa[s][i], fb[s][j], acc[i][j]);
    // every wave's DMA has landed (and every read of the other stage is done) before anyone goes
    // on; the scheduling barrier keeps the MFMAs above the wait, which the compiler would
    // otherwise hoist (they touch no memory) and so serialise the DMA with the compute
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  }

  if constexpr (EPI == EPI_STORE && sizeof(OT) == 4) {
    if (p.kslice) {                    // a K slice: plain fp32 partial tile, no bias
      GemmArgs q = p;
      q.out = reinterpret_cast<float*>(p.out) + (size_t)ks * p.split_stride;
      q.bias = nullptr;
      gemm_epilogue<OT, EPI, WM, WN>(q, acc, reinterpret_cast<float*>(smem), wave, lane, m0 + wm * WM, n0 + wn * WN);
      return;
    }
  }
  gemm_epilogue<OT, EPI, WM, WN>(p, acc, reinterpret_cast<float*>(smem), wave, lane, m0 + wm * WM, n0 + wn * WN);
}

// Sum of the K-slice partials in slice order, then the epilogue: STORE out = OT(sum + bias),
// RESID out += sum + bias (fp32).  One thread per 4 consecutive outputs.
template <typename OT, int EPI>
__global__ void __launch_bounds__(256) split_reduce_kernel(GemmArgs p, const float* __restrict__ part, int slices) {
  const long i4 = (long)blockIdx.x * 256 + threadIdx.x;
  const int n4 = p.N / 4;
  if (i4 >= (long)p.M * n4) return;
  const int m = (int)(i4 / n4), n = (int)(i4 % n4) * 4;
  const size_t stride = (size_t)p.M * p.N;
  float4 v = *reinterpret_cast<const float4*>(part + (size_t)m * p.N + n);
  for (int s = 1; s < slices; ++s) {
    const float4 w = *reinterpret_cast<const float4*>(part + s * stride + (size_t)m * p.N + n);
    v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
  }
  if (p.bias) {
    const uint2 bb = *reinterpret_cast<const uint2*>(p.bias + n);
    v.x += bf2f((bf16_t)(bb.x & 0xffff)); v.y += bf2f((bf16_t)(bb.x >> 16));
    v.z += bf2f((bf16_t)(bb.y & 0xffff)); v.w += bf2f((bf16_t)(bb.y >> 16));
  }
  if constexpr (EPI == EPI_RESID) {
    float4* o = reinterpret_cast<float4*>(reinterpret_cast<float*>(p.out) + (size_t)m * p.ldo + n);
    const float4 x = *o;
    *o = float4{x.x + v.x, x.y + v.y, x.z + v.z, x.w + v.w};
  } else {
    const float o4[4] = {v.x, v.y, v.z, v.w};
    store4<OT>(reinterpret_cast<OT*>(p.out) + (size_t)m * p.ldo + n, o4);
  }
}

template <typename TA, typename OT, int EPI, int BM, int BN, int WM, int WN>
static hipError_t launch_tile(const GemmArgs& p, hipStream_t s) {
  constexpr bool F32A = sizeof(TA) == 4;
  const size_t lds = (size_t)2 * (BM * LDK * (F32A ? 2 : 1) + BN * LDK) * sizeof(bf16_t);
  static_assert((size_t)(BM / WM) * (BN / WN) * 16 * (WN + 4) * 4 <=
                (size_t)2 * (BM * LDK + BN * LDK) * sizeof(bf16_t), "epilogue scratch exceeds the tile buffers");
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

template <typename OT, int EPI, int BM, int BN, int WM, int WN>
static hipError_t launch_dma(const GemmArgs& p, hipStream_t s, int kslices = 1) {
  constexpr size_t lds = (size_t)2 * (BM + BN) * BK * sizeof(bf16_t);
  static_assert((size_t)(BM / WM) * (BN / WN) * 16 * (WN + 4) * 4 <= lds, "epilogue scratch exceeds the stages");
  auto kern = gemm_dma_kernel<OT, EPI, BM, BN, WM, WN>;
  static bool attr_set = false;   // benign race: idempotent attribute
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int nm = (p.M + BM - 1) / BM, nn = p.N / BN;
  hipLaunchKernelGGL(kern, dim3(nm * nn * kslices), dim3((BM / WM) * (BN / WN) * 64), lds, s, p);
  return hipGetLastError();
}

// K slices for a problem whose 128x128 tiles leave most of a last round idle: slices of at least
// 1024 along K, a multiple of 64, chosen to fill whole rounds of 2 workgroups per CU best.
static int split_slices(const GemmArgs& p) {
  if (!p.split_ws) return 1;
  const long tiles = (long)((p.M + 127) / 128) * (p.N / 128);
  const long slots = 512;                         // 256 CUs, 2 workgroups each
  if (tiles >= 2 * slots) return 1;
  int best = 1;
  double best_eff = (double)tiles / (double)(((tiles + slots - 1) / slots) * slots);
  for (int sl = 2; sl <= 4; ++sl) {
    if (p.K % (64 * sl) || p.K / sl < 1024) continue;
    if ((size_t)sl * p.M * p.N > p.split_ws_floats) continue;
    const long u = tiles * sl;
    const double eff = (double)u / (double)(((u + slots - 1) / slots) * slots);
    if (eff > best_eff + 0.05) { best = sl; best_eff = eff; }
  }
  return best;
}

// The output pointer moved by (rows, cols) elements: the residual and position epilogues write
// fp32 whatever OT is.
template <typename OT, int EPI>
static void* out_at(const GemmArgs& p, size_t rows, size_t cols) {
  if constexpr (EPI == EPI_RESID || EPI == EPI_POS)
    return reinterpret_cast<float*>(p.out) + rows * p.ldo + cols;
  else
    return reinterpret_cast<OT*>(p.out) + rows * p.ldo + cols;
}

// Rows to run as 256x256 tiles ahead of the rest, which then run as 128x128 tiles (0: no split).
// With many row tiles and a last round of 256x256 tiles (one workgroup per CU) that leaves much of
// the GPU idle, the rows of whole rounds go first and the leftover rows second.  Cost in rounds of
// 256x256 tiles: leftover 128x128 tiles that fit one workgroup per CU take about half a round,
// each round of two per CU about 0.7; the split must save 0.3 of a round (the second launch's
// ramp).  The screenshot encode (53 row tiles): QKV 4 -> 3.5 rounds, MLP up 5 -> 4.5, O and down
// 2 -> 1.5; one 1008x1008 image's QKV (21 x 15 tiles): 2 -> 1.5; the 8-image MLP down (162 x 5):
// 4 -> 3.5.
static int row_split_rows(const GemmArgs& p) {
  const int nm = (p.M + 255) / 256, nn = p.N / 256;
  if (p.N % 256 || nm <= 16) return 0;
  const long tiles = (long)nm * nn, full = tiles / 256;
  if (full < 1) return 0;
  const int m1 = (int)(full * 256 / nn);
  if (m1 < 1 || m1 >= nm) return 0;
  const long rem = (long)((p.M - m1 * 256 + 127) / 128) * (p.N / 128);
  const double split = (double)(((long)m1 * nn + 255) / 256) + (rem <= 256 ? 0.5 : 0.71 * (double)((rem + 511) / 512));
  return split <= (double)((tiles + 255) / 256) - 0.3 ? m1 * 256 : 0;
}

// 128x128 tiles with K cut into split_slices(p) slices (when that is more than one): fp32 partials
// in p.split_ws, then summed in slice order by split_reduce_kernel (or left for the caller to fold,
// with p.slices_out).  *done = false when the problem runs unsplit.
template <typename OT, int EPI>
static hipError_t launch_slices128(const GemmArgs& p, hipStream_t s, bool* done) {
  *done = false;
  if constexpr (EPI == EPI_STORE || EPI == EPI_RESID) {
    const int sl = p.vt == nullptr ? split_slices(p) : 1;
    if (sl <= 1) return hipSuccess;
    *done = true;
    GemmArgs q = p;
    q.out = p.split_ws;
    q.ldo = p.N;
    q.kslice = p.K / sl;
    q.split_stride = (long)p.M * p.N;
    q.vt = nullptr;
    hipError_t e = launch_dma<float, EPI_STORE, 128, 128, 64, 64>(q, s, sl);
    if (e != hipSuccess) return e;
    if (EPI == EPI_RESID && p.slices_out != nullptr && p.bias == nullptr) {   // the caller folds them
      *p.slices_out = sl;
      return hipSuccess;
    }
    const long n4 = (long)p.M * (p.N / 4);
    hipLaunchKernelGGL((split_reduce_kernel<OT, EPI>), dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, p,
                       (const float*)p.split_ws, sl);
    return hipGetLastError();
  }
  return hipSuccess;
}

template <typename TA, typename OT, int EPI>
static hipError_t launch_epi(const GemmArgs& p, hipStream_t s) {
  if constexpr (sizeof(TA) == 2) {
    if (p.small_tiles) return launch_dma<OT, EPI, 128, 128, 64, 64>(p, s);
    if constexpr (EPI != EPI_POS) {
      if (const int m1 = row_split_rows(p)) {
        GemmArgs a = p;
        a.M = m1;
        hipError_t e = launch_dma<OT, EPI, 256, 256, 64, 128>(a, s);
        if (e != hipSuccess) return e;
        GemmArgs b = p;
        b.M = p.M - m1;
        b.A = reinterpret_cast<const bf16_t*>(p.A) + (size_t)m1 * p.lda;
        b.out = out_at<OT, EPI>(p, m1, 0);
        b.vt_row0 = p.vt_row0 + m1;
        // the leftover rows are few tiles (a 1092x2408 screenshot's O and down projections: 30 of
        // 128x128): with a long K they take K slices (its down projection: 4, 120 workgroups)
        if (p.slices_out == nullptr) {
          bool done = false;
          const hipError_t e2 = launch_slices128<OT, EPI>(b, s, &done);
          if (done || e2 != hipSuccess) return e2;
        }
        return launch_dma<OT, EPI, 128, 128, 64, 64>(b, s);
      }
    }
  }
  // 256x256 tiles with 8 waves (two per SIMD, each 64x128) when there are at least two tiles per
  // CU; otherwise 128x128 tiles with 4 waves (two workgroups per CU), with K split into slices
  // when those tiles cannot fill the GPU (and the caller gave a workspace).  A projection that
  // also stores V^T (p.vt) always runs as one launch: the split paths have no V^T epilogue.
  if constexpr (sizeof(TA) == 2 && (EPI == EPI_STORE || EPI == EPI_RESID)) {
    const long tiles256 = (long)((p.M + 255) / 256) * (p.N / 256);
    // a very long K whose 256x256 tiles make one round of at least three quarters of the GPU
    // (the 3.6k-token prefill's down projection: 14 x 14 tiles, K = 18944): one unsplit launch,
    // without the split partials' traffic
    if (p.N % 256 == 0 && p.K >= 8192 && tiles256 >= 192 && tiles256 <= 256)
      return launch_dma<OT, EPI, 256, 256, 64, 128>(p, s);
    // a long K whose 256x256 tiles fill under three quarters of the GPU (the 1500-token prefill's
    // down projection: 6 x 14 tiles, K = 18944; its O projection: 6 x 14 tiles, K = 3584): K
    // slices of 256x256 tiles that make one round of at least 224 of the 256 CUs (3 slices of
    // 6336, 6336 and 6272, and of 1216, 1216 and 1152 there), then the fp32 partials summed in
    // slice order
    if (p.split_ws && p.vt == nullptr && p.N % 256 == 0 && p.K >= 3072 && tiles256 < 192) {
      int sl = 0;
      for (int c = 2; c <= 4 && !sl; ++c) {
        const int kslice = (p.K / BK + c - 1) / c * BK;
        if (tiles256 * c >= 224 && tiles256 * c <= 256 && p.K - (c - 1) * kslice >= 1024 &&
            (size_t)c * p.M * p.N <= p.split_ws_floats)
          sl = c;
      }
      if (sl) {
        GemmArgs q = p;
        q.out = p.split_ws;
        q.ldo = p.N;
        q.kslice = (p.K / BK + sl - 1) / sl * BK;
        q.split_stride = (long)p.M * p.N;
        q.vt = nullptr;
        hipError_t e = launch_dma<float, EPI_STORE, 256, 256, 64, 128>(q, s, sl);
        if (e != hipSuccess) return e;
        if (EPI == EPI_RESID && p.slices_out != nullptr && p.bias == nullptr) {   // the caller folds them
          *p.slices_out = sl;
          return hipSuccess;
        }
        const long n4 = (long)p.M * (p.N / 4);
        hipLaunchKernelGGL((split_reduce_kernel<OT, EPI>), dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, p,
                           (const float*)p.split_ws, sl);
        return hipGetLastError();
      }
    }
    // 256x256 tiles that fill at least three quarters of one round of the GPU (one workgroup per
    // CU) beat two rounds of 128x128 tiles (the 3.6k-token prefill's QKV projection: 14 x 18
    // tiles, 157 -> 99 us; the one-image encode's MLP up projection)
    if (p.N % 256 == 0 && tiles256 >= 192 && tiles256 < 512) return launch_dma<OT, EPI, 256, 256, 64, 128>(p, s);
    if (!(p.N % 256 == 0 && tiles256 >= 512) && p.vt == nullptr) {
      bool done = false;
      const hipError_t e = launch_slices128<OT, EPI>(p, s, &done);
      if (done || e != hipSuccess) return e;
    }
  }
  if constexpr (sizeof(TA) == 2) {
    const int nm = (p.M + 255) / 256;
    const long tiles = (long)nm * (p.N / 256);
    if (p.N % 256 == 0 && tiles >= 512) {
      // few row tiles and many column tiles (the prefill's gate/up projection: 6 x 148): the
      // columns of whole rounds of 256x256 tiles, then the rest with 128x128 tiles, so that the
      // last round is not left mostly idle
      const long rounds = tiles / 256;
      const int n1 = (int)(rounds * 256 / nm) * 256;
      if (tiles % 256 >= 32 && nm <= 16 && n1 < p.N && EPI != EPI_POS && p.vt == nullptr) {
        GemmArgs a = p;
        a.N = n1;
        hipError_t e = launch_dma<OT, EPI, 256, 256, 64, 128>(a, s);
        if (e != hipSuccess) return e;
        GemmArgs b = p;
        b.N = p.N - n1;
        b.W = p.W + (size_t)n1 * p.ldw;
        if (p.bias) b.bias = p.bias + n1;
        b.out = out_at<OT, EPI>(p, 0, EPI == EPI_SWIGLU ? n1 / 2 : n1);
        return launch_dma<OT, EPI, 128, 128, 64, 64>(b, s);
      }
      return launch_dma<OT, EPI, 256, 256, 64, 128>(p, s);
    }
    if (p.N % 256 == 0 && tiles >= 192) return launch_dma<OT, EPI, 256, 256, 64, 128>(p, s);
    return launch_dma<OT, EPI, 128, 128, 64, 64>(p, s);
  }
  return launch_tile<TA, OT, EPI, 128, 128, 64, 64>(p, s);
}

template <typename TA, typename OT>
hipError_t gemm(const GemmArgs& p, int epi, hipStream_t s) {
  if (p.slices_out != nullptr) *p.slices_out = 0;
  if (p.M <= 0) return hipSuccess;
  if (p.N % 128 || p.K % BK || p.lda % 8 || p.ldw % 8 || p.ldo % 4) return hipErrorInvalidValue;
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
