// Flash-style attention for vision encode (bidirectional) and LLM prefill (causal, grouped-query).
//
// softmax(q k^T / sqrt(d)) v is computed tile by tile with an online softmax in fp32 (the
// attention kernel of the paper's Table 3; the paper used FlashInfer, Sec. 4).  gfx950 design:
//  * a workgroup owns 128 queries of one head (4 waves x 32); K and V^T tiles of 64 keys are
//    staged in LDS and shared by the 4 waves; the next tile is prefetched into registers while
//    the current one is consumed;
//  * S^T = K Q^T with MFMA 32x32x16 so that each lane owns ONE query (column) and 16 keys:
//    the row max / row sum need a single cross-lane exchange (lane ^ 32), and the output
//    rescale is per lane;
//  * O^T = V^T P^T with the same MFMA: the probabilities already sit in the B-operand layout,
//    because an MFMA fragment's k index only has to agree between its A and B operands;
//    V is therefore stored transposed by the projection kernel, and each V^T tile row is
//    stored with two 4-key blocks of every 16 swapped so that a fragment is one 16-byte read;
//  * head_dim 64 / 80 / 128 (80 = 5 k-steps of 16 for QK^T; PV pads the output rows to 96);
//  * fp32 mode (tiny-stack exact mode): q, k, v, p are split into bf16 hi + lo parts and the
//    three significant cross products are accumulated;
//  * bidirectional bf16 with head_dim <= 80 (the vision encoder) runs a wider variant: two query
//    groups per wave share every fragment read, and the row sums come out of the P V^T MFMAs;
//  * causal: when all (head, query block) workgroups fit in one round of workgroup slots, the
//    heaviest blocks are cut into key ranges whose fp32 partials the last range to finish merges,
//    so the longest chain of key tiles is not the whole sequence.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace nova {

constexpr int AQ = 128;   // queries per workgroup
constexpr int AK = 64;    // keys per tile

// Combine a value with that of lane ^ 32 (the other half of the wavefront holds the same query
// columns of a 32x32 MFMA tile): gfx950's permlane32 swap exchanges the two halves in the VALU,
// without the LDS round trip of a general shuffle.  Swapping x with itself gives, in every lane,
// x of that lane and of its partner.
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// NW waves of 32 queries per workgroup (4 on every path)
template <typename T, int D, bool CAUSAL, int NW>
__global__ void __launch_bounds__(NW * 64, 2) attn_kernel(AttnArgs p) {
  constexpr int AQB = NW * 32;              // queries per workgroup
  constexpr int NT = NW * 64;               // threads per workgroup
  constexpr bool F32 = sizeof(T) == 4;
  constexpr int NS = D / 16;                // k-steps of QK^T
  constexpr int DP = (D + 31) / 32 * 32;    // output rows padded to 32
  constexpr int NC = DP / 32;               // output row blocks
  constexpr int KP = D + 8;                 // LDS pitch of K rows (bf16)
  constexpr int VP = AK + 8;                // LDS pitch of V^T rows (bf16, 16-byte aligned rows)
  constexpr int NPART = F32 ? 2 : 1;
  __shared__ __align__(16) bf16_t ks[NPART][AK * KP];
  __shared__ __align__(16) bf16_t vs[NPART][DP * VP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5, lq = lane & 31;
  const int nqb = (p.sq + AQB - 1) / AQB;
  // one-dimensional grid: workgroups are dealt to the 8 XCDs round-robin, so when the (batch,
  // head) pairs split evenly over the XCDs each XCD takes whole pairs, one after another, and the
  // pair's K and V stay in its L2 while all of the pair's query blocks read them
  int qbi, h, b;
  int pair, part = 0, nparts = 1, slot = 0;
  {
    const int pairs = p.batch * p.n_q;
    int lin = blockIdx.x;
    if (CAUSAL && p.kv_tmax > 0) {
      // key ranges: query block q is cut into P(q) = ceil(tiles(q) / kv_tmax) ranges of whole
      // tiles.  The grid runs level by level from the heaviest block down, each level holding
      // every pair's ranges of that block (range-major); a multi-range block's partials take
      // P(q) consecutive slots of its pair's kv_slots
      int units = 0, slots = 0, q = nqb - 1, P = 1;
      for (;; --q) {
        P = ((min(p.sk, (q + 1) * AQB) + AK - 1) / AK + p.kv_tmax - 1) / p.kv_tmax;
        if (lin < (units + P) * pairs || q == 0) break;
        units += P;
        if (P > 1) slots += P;
      }
      lin -= units * pairs;
      qbi = nqb - 1 - q;
      nparts = P;
      part = lin / pairs;
      pair = lin - part * pairs;
      slot = pair * p.kv_slots + p.kv_slots - slots - (P > 1 ? P : 0) + part;
    } else if (CAUSAL) {
      // heaviest blocks of every head first: the workgroups dispatched last, which share a CU
      // with an earlier one, are the lightest; head h's blocks fall on XCDs (h + pairs k) % 8
      qbi = lin / pairs;
      pair = lin % pairs;
    } else if (pairs % 8 == 0) {
      const int j = lin >> 3;
      pair = (lin & 7) * (pairs >> 3) + j / nqb;
      qbi = j % nqb;
    } else {
      pair = lin / nqb;
      qbi = lin % nqb;
    }
    h = pair % p.n_q;
    b = pair / p.n_q;
  }
  const int qb = CAUSAL ? (nqb - 1 - qbi) : qbi;   // heavy causal blocks first
  const int kvh = h / (p.n_q / p.n_kv);
  const int q0 = qb * AQB;
  const int qrow = q0 + wave * 32 + lq;

  const T* Q = reinterpret_cast<const T*>(p.q) + (size_t)b * p.q_batch + (size_t)h * D;
  const T* K = reinterpret_cast<const T*>(p.k) + (size_t)b * p.k_batch + (size_t)kvh * D;
  const T* VT = reinterpret_cast<const T*>(p.vt) + ((size_t)b * p.n_kv + kvh) * D * (size_t)p.sk_pad;

  // ---- Q fragments (B operand of S^T = K Q^T): query lq, dims 16s + 8g .. +8
  Frag8 qh[NS], ql[F32 ? NS : 1];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if (qrow < p.sq) {
      const T* src = Q + (size_t)qrow * p.q_row + 16 * s + 8 * g;
      if constexpr (F32) {
        float x[8];
        *reinterpret_cast<float4*>(x) = *reinterpret_cast<const float4*>(src);
        *reinterpret_cast<float4*>(x + 4) = *reinterpret_cast<const float4*>(src + 4);
        split8(x, qh[s], ql[s]);
      } else {
        qh[s] = *reinterpret_cast<const Frag8*>(src);
      }
    } else {
      qh[s] = zero_frag();
      if constexpr (F32) ql[s] = zero_frag();
    }
  }

  // ---- tile staging (global -> registers -> LDS)
  constexpr int EPC = F32 ? 4 : 8;                     // elements per 16-byte chunk
  constexpr int K_CH = AK * D / EPC;
  constexpr int V_CH = D * AK / EPC;
  constexpr int K_IT = (K_CH + NT - 1) / NT, V_IT = (V_CH + NT - 1) / NT;
  u32x4 rk[K_IT], rv[V_IT];
  // loads are unconditional (chunk index and key row clamped) so that the waits for them stay
  // exact; the surplus chunks are never stored and keys past sk are masked
  auto load_tile = [&](int kv0) {
#pragma unroll
    for (int i = 0; i < K_IT; ++i) {
      const int c = min(tid + i * NT, K_CH - 1);
      const int r = c / (D / EPC), col = (c % (D / EPC)) * EPC;
      rk[i] = *reinterpret_cast<const u32x4*>(K + (size_t)min(kv0 + r, p.sk - 1) * p.k_row + col);
    }
#pragma unroll
    for (int i = 0; i < V_IT; ++i) {
      const int c = min(tid + i * NT, V_CH - 1);
      const int r = c / (AK / EPC), col = (c % (AK / EPC)) * EPC;
      rv[i] = *reinterpret_cast<const u32x4*>(VT + (size_t)r * p.sk_pad + kv0 + col);
    }
  };
  // V^T tiles keep each row's keys in groups of 16 with the middle two 4-key blocks swapped
  // (block b at position 2 (b % 2) + b / 2): the 8 keys a lane's P fragment covers, 4 at 4g and 4
  // at 8 + 4g, then sit side by side and the A fragment is one 16-byte read
  auto vpos = [](int key) { const int b = (key >> 2) & 3; return (key & ~15) + 4 * (((b & 1) << 1) | (b >> 1)); };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < K_IT; ++i) {
      const int c = tid + i * NT;
      if (c < K_CH) {
        const int r = c / (D / EPC), col = (c % (D / EPC)) * EPC;
        if constexpr (F32) {
          float x[4] = {__uint_as_float(rk[i][0]), __uint_as_float(rk[i][1]), __uint_as_float(rk[i][2]), __uint_as_float(rk[i][3])};
          bf16_t hh[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) hh[j] = f2bf(x[j]);
          *reinterpret_cast<uint2*>(&ks[0][r * KP + col]) =
              make_uint2((uint32_t)hh[0] | ((uint32_t)hh[1] << 16), (uint32_t)hh[2] | ((uint32_t)hh[3] << 16));
          *reinterpret_cast<uint2*>(&ks[1][r * KP + col]) =
              make_uint2(pack2(x[0] - bf2f(hh[0]), x[1] - bf2f(hh[1])), pack2(x[2] - bf2f(hh[2]), x[3] - bf2f(hh[3])));
        } else {
          *reinterpret_cast<u32x4*>(&ks[0][r * KP + col]) = rk[i];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < V_IT; ++i) {
      const int c = tid + i * NT;
      if (c < V_CH) {
        const int r = c / (AK / EPC), col = (c % (AK / EPC)) * EPC;
        if constexpr (F32) {
          float x[4] = {__uint_as_float(rv[i][0]), __uint_as_float(rv[i][1]), __uint_as_float(rv[i][2]), __uint_as_float(rv[i][3])};
          bf16_t hh[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) hh[j] = f2bf(x[j]);
          *reinterpret_cast<uint2*>(&vs[0][r * VP + vpos(col)]) =
              make_uint2((uint32_t)hh[0] | ((uint32_t)hh[1] << 16), (uint32_t)hh[2] | ((uint32_t)hh[3] << 16));
          *reinterpret_cast<uint2*>(&vs[1][r * VP + vpos(col)]) =
              make_uint2(pack2(x[0] - bf2f(hh[0]), x[1] - bf2f(hh[1])), pack2(x[2] - bf2f(hh[2]), x[3] - bf2f(hh[3])));
        } else {
          *reinterpret_cast<uint2*>(&vs[0][r * VP + vpos(col)]) = make_uint2(rv[i][0], rv[i][1]);
          *reinterpret_cast<uint2*>(&vs[0][r * VP + vpos(col + 4)]) = make_uint2(rv[i][2], rv[i][3]);
        }
      }
    }
  };

  f32x16 o[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) o[c] = f32x16{};
  float m_run = -1e30f, l_run = 0.f;
  const float scale = 1.4426950408889634f / sqrtf((float)D);

  const int kv_end = CAUSAL ? min(p.sk, q0 + AQB) : p.sk;
  int kv_lo = 0, kv_hi = kv_end;
  if (CAUSAL && nparts > 1) {     // this workgroup's range: whole tiles, as even as they split
    const int per = ((kv_end + AK - 1) / AK + nparts - 1) / nparts;
    kv_lo = part * per * AK;
    kv_hi = min(kv_end, kv_lo + per * AK);
  }
  const int wave_qmax = q0 + wave * 32 + 31;
  load_tile(kv_lo);
  for (int kv0 = kv_lo; kv0 < kv_hi; kv0 += AK) {
    __syncthreads();          // previous tile fully consumed
    store_tile();
    __syncthreads();
    if (kv0 + AK < kv_hi) load_tile(kv0 + AK);
    if (CAUSAL && kv0 > wave_qmax) continue;   // every key of this tile is in this wave's future

    // S^T = K Q^T for two 32-key blocks
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int off = (kb * 32 + lq) * KP + 16 * s + 8 * g;
        Frag8 ka = *reinterpret_cast<const Frag8*>(&ks[0][off]);
        sacc[kb] = mfma32(ka, qh[s], sacc[kb]);
        if constexpr (F32) {
          Frag8 kl = *reinterpret_cast<const Frag8*>(&ks[1][off]);
          sacc[kb] = mfma32(kl, qh[s], sacc[kb]);
          sacc[kb] = mfma32(ka, ql[s], sacc[kb]);
        }
      }
    }
    // online softmax for query qrow over keys kv0 + 32kb + 8(r/4) + 4g + r%4; the running max is
    // kept in raw score units and the 1/sqrt(d) scale is folded into the exp2 argument.
    const bool need_mask = (kv0 + AK > p.sk) || (CAUSAL && kv0 + AK - 1 > q0 + wave * 32);
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kidx = kv0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          const bool ok = kidx < p.sk && (!CAUSAL || kidx <= qrow);
          sacc[kb][r] = ok ? sacc[kb][r] : -INFINITY;
        }
    }
    float tmax = -1e30f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, sacc[kb][r]);
    tmax = max_halves(tmax);
    const float m_new = fmaxf(m_run, tmax);
    const float ms = m_new * scale;
    float rsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[kb][r], scale, -ms));
        sacc[kb][r] = pv;
        rsum += pv;
      }
    rsum = sum_halves(rsum);
    if (__ballot(m_new > m_run)) {       // rescale only when some query's max moved
      const float corr = __builtin_amdgcn_exp2f((m_run - m_new) * scale);
      l_run *= corr;
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[c][r] *= corr;
    }
    l_run += rsum;
    m_run = m_new;

    // O^T += V^T P^T, 16 keys per MFMA
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        Frag8 ph, pl;
        if constexpr (F32) {
          float x[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = sacc[kb][8 * t + e];
          split8(x, ph, pl);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) ph.w[e] = pack2(sacc[kb][8 * t + 2 * e], sacc[kb][8 * t + 2 * e + 1]);
        }
        const int kpos = kb * 32 + 16 * t + 8 * g;     // keys 16t + 4g + 0..3 and 16t + 8 + 4g + 0..3
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const int vrow = c * 32 + lq;
          const Frag8 va = *reinterpret_cast<const Frag8*>(&vs[0][vrow * VP + kpos]);
          o[c] = mfma32(va, ph, o[c]);
          if constexpr (F32) {
            const Frag8 vl = *reinterpret_cast<const Frag8*>(&vs[1][vrow * VP + kpos]);
            o[c] = mfma32(vl, ph, o[c]);
            o[c] = mfma32(va, pl, o[c]);
          }
        }
      }
  }

  if (CAUSAL && nparts > 1) {
    // Every range stores its unnormalised output, running max and sum (fp32, [value][thread] per
    // slot) with device-scope atomic stores, written through to the coherent level; every thread
    // waits until its stores are acknowledged there before the workgroup barrier, and only then
    // does thread 0 count the range in.  The last range of the block to arrive reads the others
    // back with device-scope atomic loads and merges all of them in range order, so the result
    // does not depend on which range finished last.
    constexpr int PV = NC * 16 + 2;
    float* po = reinterpret_cast<float*>(p.part);
    auto at = [&](int sl, int v) { return po + ((size_t)sl * PV + v) * NT + tid; };
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) __hip_atomic_store(at(slot, c * 16 + r), o[c][r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(at(slot, NC * 16), m_run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(at(slot, NC * 16 + 1), l_run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __shared__ int last;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    unsigned* cnt = p.counters + (size_t)pair * nqb + qb;
    if (tid == 0) last = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(nparts - 1);
    __syncthreads();
    if (!last) return;
    if (tid == 0) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int s0 = slot - part;
    float mk[8], mmax = -1e30f;       // at most 8 ranges (the launcher's bound)
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      mk[k] = k >= nparts ? -1e30f : k == part ? m_run : __hip_atomic_load(at(s0 + k, NC * 16), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      mmax = fmaxf(mmax, mk[k]);
    }
    f32x16 acc[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[c] = f32x16{};
    float lsum = 0.f;
    for (int k = 0; k < nparts; ++k) {
      float w = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) w = j == k ? mk[j] : w;
      w = __builtin_amdgcn_exp2f((w - mmax) * scale);
      if (k == part) {
        lsum += w * l_run;
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[c][r] += w * o[c][r];
      } else {
        lsum += w * __hip_atomic_load(at(s0 + k, NC * 16 + 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        float t[NC][16];
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) t[c][r] = __hip_atomic_load(at(s0 + k, c * 16 + r), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[c][r] += w * t[c][r];
      }
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) o[c] = acc[c];
    l_run = lsum;
  }

  if (qrow >= p.sq) return;
  const float inv = 1.0f / l_run;
  T* out = reinterpret_cast<T*>(p.out) + (size_t)b * p.o_batch + (size_t)qrow * p.o_row + (size_t)h * D;
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int col = c * 32 + 8 * r4 + 4 * g;
      if (col >= D) continue;
      if constexpr (F32) {
        *reinterpret_cast<float4*>(out + col) =
            make_float4(o[c][4 * r4] * inv, o[c][4 * r4 + 1] * inv, o[c][4 * r4 + 2] * inv, o[c][4 * r4 + 3] * inv);
      } else {
        *reinterpret_cast<uint2*>(out + col) =
            make_uint2(pack2(o[c][4 * r4] * inv, o[c][4 * r4 + 1] * inv), pack2(o[c][4 * r4 + 2] * inv, o[c][4 * r4 + 3] * inv));
      }
    }
}

// Bidirectional bf16 attention with two 32-query groups per wave (256 queries per workgroup):
// each K and V^T fragment read from LDS feeds two MFMAs, and each K/V tile the workgroup stages
// serves twice the queries, which halves the LDS and L2 traffic per flop of the kernel above.
//  * K and V^T tiles go global -> LDS by 16-byte LDS-DMA loads into two stages (separate arrays,
//    the loop unrolled by two so that each stage is addressed statically): the next tile loads
//    while this one is consumed, with one barrier per tile and no staging registers;
//  * the K rows of every 16-key group are stored with their middle two 4-row blocks swapped.
//    The S^T accumulator rows a lane holds are then keys 16t + 8g .. +7 of chunk t, in order,
//    which is the k range of the P^T operand, so the V^T tile is used in natural key order;
//  * when the head dimension is padded up to the 32-row MFMA block (d = 80 -> 96), the padding
//    rows of the V^T tiles hold ones, so the P V^T product also accumulates each query's sum of
//    (bf16) probabilities, rescaled together with the output: no separate row sum is kept.
constexpr int AQW = 256;

__device__ __forceinline__ void attn_dma16(const bf16_t* g, bf16_t* l_base) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)l_base, 16, 0, 0);
}

// Light-block sweep of attn_wide_kernel: one 32-key step of one query group.  Row i of the score
// accumulator holds key perm(i) (the middle 4-row blocks of each 16 swapped, as in the LDS tiles),
// so a lane's probabilities of chunk tt are keys 16 tt + 8 g .. + 7 in order.
template <int D, int NS, int NC, bool ONES>
__device__ __forceinline__ void light_step(const Frag8 (&q1)[NS], const Frag8 (&kf)[NS], const Frag8 (&vf)[2][NC],
                                           int key0, int sk, int g, float scale, f32x16 (&o1)[NC], float& m1,
                                           float& l1) {
  f32x16 sacc = f32x16{};
#pragma unroll
  for (int s = 0; s < NS; ++s) sacc = mfma32(kf[s], q1[s], sacc);
  if (key0 + 32 > sk) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (key0 + 16 * (r >> 3) + 8 * g + (r & 7) >= sk) sacc[r] = -INFINITY;
  }
  float tmax = -1e30f;
#pragma unroll
  for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, sacc[r]);
  tmax = max_halves(tmax);
  const float m_new = fmaxf(m1, tmax);
  const float ms = m_new * scale;
  float rsum = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[r], scale, -ms));
    sacc[r] = pv;
    if constexpr (!ONES) rsum += pv;
  }
  if (__ballot(m_new > m1)) {
    const float corr = __builtin_amdgcn_exp2f((m1 - m_new) * scale);
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) o1[c][r] *= corr;
    if constexpr (!ONES) l1 *= corr;
  }
  if constexpr (!ONES) l1 += sum_halves(rsum);
  m1 = m_new;
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    Frag8 ph;
#pragma unroll
    for (int e = 0; e < 4; ++e) ph.w[e] = pack2(sacc[8 * tt + 2 * e], sacc[8 * tt + 2 * e + 1]);
#pragma unroll
    for (int c = 0; c < NC; ++c) o1[c] = mfma32(vf[tt][c], ph, o1[c]);
  }
}

template <int D>
__global__ void __launch_bounds__(256, 2) attn_wide_kernel(AttnArgs p) {
  constexpr int NS = D / 16;
  constexpr int DP = (D + 31) / 32 * 32;
  constexpr int NC = DP / 32;
  constexpr int KP = D + 8, VP = AK + 8;
  constexpr int KPS = KP / 8, VPS = VP / 8;            // 16-byte slots per LDS row (last one: pad)
  constexpr int K_INS = (AK * KPS + 63) / 64, V_INS = (D * VPS + 63) / 64;
  constexpr int K_IW = (K_INS + 3) / 4, V_IW = (V_INS + 3) / 4;   // DMA instructions per wave
  constexpr bool ONES = DP > D;
  __shared__ __align__(16) bf16_t ks0[AK * KP];
  __shared__ __align__(16) bf16_t vs0[DP * VP];
  __shared__ __align__(16) bf16_t ks1[AK * KP];
  __shared__ __align__(16) bf16_t vs1[DP * VP];

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, lq = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // scalar: uniform branches
  const int nqb = (p.sq + AQW - 1) / AQW;
  // A last query block of at most 64 queries ("light") would keep three of its four waves idle
  // for a whole key sweep and, with every other block full, add a round of workgroups at the end
  // (8 images of 5184 patches: 20 full blocks and one of 64 queries per head).  Light blocks are
  // dispatched first; each of their waves takes one query group and one 32-key half of every tile.
  const bool has_light = p.sq % AQW != 0 && p.sq % AQW <= 64;
  const int pairs = p.batch * p.n_q;
  // key range: with kv_parts > 1, workgroup blockIdx.x takes range blockIdx.x / (workgroups of
  // one range) of whole 64-key tiles, the same (query block, head) layout in every range
  const int kpart = blockIdx.x / (nqb * pairs);
  const int tpp = ((p.sk + AK - 1) / AK + p.kv_parts - 1) / p.kv_parts;
  const int kbeg = min(kpart * tpp * AK, p.sk), kend = min((kpart + 1) * tpp * AK, p.sk);
  int qb, h, b;
  bool light = false;
  {
    const int lin = blockIdx.x - kpart * nqb * pairs;
    int pair;
    if (has_light && lin < pairs) {
      light = true;
      qb = nqb - 1;
      // a pair's light block on the XCD of its full blocks (same L2)
      pair = pairs % 8 == 0 ? (lin & 7) * (pairs >> 3) + (lin >> 3) : lin;
    } else {
      const int lin2 = lin - (has_light ? pairs : 0), nfull = has_light ? nqb - 1 : nqb;
      if (pairs % 8 == 0) {
        const int j = lin2 >> 3;
        pair = (lin2 & 7) * (pairs >> 3) + j / nfull;
        qb = j % nfull;
      } else {
        pair = lin2 / nfull;
        qb = lin2 % nfull;
      }
    }
    h = pair % p.n_q;
    b = pair / p.n_q;
  }
  const int kvh = h / (p.n_q / p.n_kv);
  const int qbase = qb * AQW + wave * 64;          // group u holds queries qbase + 32 u + lq
  const bool active = qbase < p.sq;

  const bf16_t* Q = reinterpret_cast<const bf16_t*>(p.q) + (size_t)b * p.q_batch + (size_t)h * D;
  const bf16_t* K = reinterpret_cast<const bf16_t*>(p.k) + (size_t)b * p.k_batch + (size_t)kvh * D;
  const bf16_t* VT = reinterpret_cast<const bf16_t*>(p.vt) + ((size_t)b * p.n_kv + kvh) * D * (size_t)p.sk_pad;

  const float scale = 1.4426950408889634f / sqrtf((float)D);
  // where a query row's normalised output goes: the output itself, or with several key ranges
  // this range's partial row (bf16, [range][pair][query][D]) and its (max, sum) (fp32 pairs after
  // all partial rows), written by the lanes of the first half
  auto out_row = [&](int bb, int hh, int qrow, float m, float lsum) -> bf16_t* {
    if (p.kv_parts == 1)
      return reinterpret_cast<bf16_t*>(p.out) + (size_t)bb * p.o_batch + (size_t)qrow * p.o_row + (size_t)hh * D;
    const size_t row = ((size_t)kpart * pairs + (size_t)bb * p.n_q + hh) * p.sq + qrow;
    bf16_t* po = reinterpret_cast<bf16_t*>(p.part);
    if (g == 0) reinterpret_cast<float2*>(po + (size_t)p.kv_parts * pairs * p.sq * D)[row] = make_float2(m, lsum);
    return po + row * D;
  };
  // DMA instruction i (dealt to wave i % 4) fills LDS slots 64 i .. 64 i + 63 of a tile, slot j
  // being piece j % (slots per row) of LDS row j / (slots per row); pad slots are masked off
  int k_row[K_IW], k_col[K_IW], v_off[V_IW];
  bool k_on[K_IW], v_on[V_IW];
#pragma unroll
  for (int t = 0; t < K_IW; ++t) {
    const int ins = wave + 4 * t, j = ins * 64 + lane, r = j / KPS, pc = j % KPS;
    k_on[t] = ins < K_INS && pc < KPS - 1;
    k_row[t] = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);     // key of LDS row r
    k_col[t] = pc * 8;
  }
#pragma unroll
  for (int t = 0; t < V_IW; ++t) {
    const int ins = wave + 4 * t, j = ins * 64 + lane, r = j / VPS, pc = j % VPS;
    v_on[t] = ins < V_INS && pc < VPS - 1 && r < D;
    v_off[t] = r * p.sk_pad + pc * 8;
  }
  auto dma = [&](int kv0, bf16_t* kl, bf16_t* vl) {
#pragma unroll
    for (int t = 0; t < K_IW; ++t)
      if (k_on[t]) attn_dma16(K + (size_t)min(kv0 + k_row[t], p.sk - 1) * p.k_row + k_col[t], kl + (wave + 4 * t) * 512);
#pragma unroll
    for (int t = 0; t < V_IW; ++t)
      if (v_on[t]) attn_dma16(VT + v_off[t] + kv0, vl + (wave + 4 * t) * 512);
  };
  if constexpr (ONES) {       // rows D .. DP-1 of both V^T stages: bf16 ones, never overwritten
    for (int i = tid; i < (DP - D) * VP / 2; i += 256) {
      reinterpret_cast<uint32_t*>(vs0 + D * VP)[i] = 0x3f803f80u;
      reinterpret_cast<uint32_t*>(vs1 + D * VP)[i] = 0x3f803f80u;
    }
  }

  if (light) {
    // wave w: key half w & 1 of every 64-key tile and query group w >> 1 of the block's 64 queries;
    // K and V^T tiles come through the same double-buffered DMA stages as for a full block, each
    // wave doing a quarter of a full wave's MFMAs per tile.  The two key halves of a query group
    // are merged through LDS at the end.
    const int kb = wave & 1, u = wave >> 1;
    const int qrow = qb * AQW + 32 * u + lq;
    const bool lact = qb * AQW + 32 * u < p.sq;
    Frag8 q1[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s)
      q1[s] = qrow < p.sq ? *reinterpret_cast<const Frag8*>(Q + (size_t)qrow * p.q_row + 16 * s + 8 * g) : zero_frag();
    f32x16 o1[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) o1[c] = f32x16{};
    float m1 = -1e30f, l1 = 0.f;
    auto ltile = [&](int kv0, const bf16_t* ks, const bf16_t* vs) {
      Frag8 kf[NS], vf[2][NC];
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[s] = *reinterpret_cast<const Frag8*>(&ks[(kb * 32 + lq) * KP + 16 * s + 8 * g]);
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int c = 0; c < NC; ++c)
          vf[tt][c] = *reinterpret_cast<const Frag8*>(&vs[(c * 32 + lq) * VP + kb * 32 + 16 * tt + 8 * g]);
      light_step<D, NS, NC, ONES>(q1, kf, vf, kv0 + 32 * kb, p.sk, g, scale, o1, m1, l1);
    };
    dma(kbeg, ks0, vs0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int kv0 = kbeg; kv0 < kend; kv0 += 2 * AK) {
      if (kv0 + AK < kend) dma(kv0 + AK, ks1, vs1);
      if (lact) ltile(kv0, ks0, vs0);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (kv0 + AK >= kend) break;
      if (kv0 + 2 * AK < kend) dma(kv0 + 2 * AK, ks0, vs0);
      if (lact) ltile(kv0 + AK, ks1, vs1);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
    // the second-half wave of group u leaves (o, m, l) in V^T stage u (every tile read is done),
    // the first-half wave combines them and writes the output
    constexpr int CW = NC * 16 + 2;                     // floats per lane
    static_assert((size_t)CW * 64 * 4 <= sizeof(vs0), "merge buffer");
    float* cb = reinterpret_cast<float*>(u ? vs1 : vs0);
    if (kb) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) cb[(c * 16 + r) * 64 + lane] = o1[c][r];
      cb[(NC * 16) * 64 + lane] = m1;
      cb[(NC * 16 + 1) * 64 + lane] = l1;
    }
    __syncthreads();
    if (kb || qrow >= p.sq) return;
    const float m2 = cb[(NC * 16) * 64 + lane], l2 = cb[(NC * 16 + 1) * 64 + lane];
    const float mm = fmaxf(m1, m2);
    const float f1 = __builtin_amdgcn_exp2f((m1 - mm) * scale), f2 = __builtin_amdgcn_exp2f((m2 - mm) * scale);
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) o1[c][r] = o1[c][r] * f1 + cb[(c * 16 + r) * 64 + lane] * f2;
    const float lsum = ONES ? o1[NC - 1][8] : l1 * f1 + l2 * f2;
    const float inv = 1.0f / lsum;
    bf16_t* out = out_row(b, h, qrow, mm, lsum);
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + 8 * r4 + 4 * g;
        if (col >= D) continue;
        *reinterpret_cast<uint2*>(out + col) =
            make_uint2(pack2(o1[c][4 * r4] * inv, o1[c][4 * r4 + 1] * inv), pack2(o1[c][4 * r4 + 2] * inv, o1[c][4 * r4 + 3] * inv));
      }
    return;
  }

  Frag8 qh[2][NS];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int qrow = qbase + 32 * u + lq;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qh[u][s] = qrow < p.sq ? *reinterpret_cast<const Frag8*>(Q + (size_t)qrow * p.q_row + 16 * s + 8 * g) : zero_frag();
  }

  f32x16 o[2][NC];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int c = 0; c < NC; ++c) o[u][c] = f32x16{};
  float m_run[2] = {-1e30f, -1e30f}, l_run[2] = {0.f, 0.f};

  auto tile = [&](int kv0, const bf16_t* ks, const bf16_t* vs) {
    // the online softmax advances 32 keys at a time: half the score registers, and the next
    // block's S^T MFMAs are independent of this block's exponentials
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const Frag8 ka = *reinterpret_cast<const Frag8*>(&ks[(kb * 32 + lq) * KP + 16 * s + 8 * g]);
        sacc[0] = mfma32(ka, qh[0][s], sacc[0]);
        sacc[1] = mfma32(ka, qh[1][s], sacc[1]);
      }
      // element r of a lane is key kv0 + 32 kb + 16 (r / 8) + 8 g + r % 8
      if (kv0 + kb * 32 + 32 > p.sk) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (kv0 + kb * 32 + 16 * (r >> 3) + 8 * g + (r & 7) >= p.sk) sacc[u][r] = -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float tmax = -1e30f;
#pragma unroll
        for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, sacc[u][r]);
        tmax = max_halves(tmax);
        const float m_new = fmaxf(m_run[u], tmax);
        const float ms = m_new * scale;
        float rsum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[u][r], scale, -ms));
          sacc[u][r] = pv;
          if constexpr (!ONES) rsum += pv;
        }
        if (__ballot(m_new > m_run[u])) {
          const float corr = __builtin_amdgcn_exp2f((m_run[u] - m_new) * scale);
#pragma unroll
          for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[u][c][r] *= corr;
          if constexpr (!ONES) l_run[u] *= corr;
        }
        if constexpr (!ONES) l_run[u] += sum_halves(rsum);
        m_run[u] = m_new;
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        Frag8 ph[2];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e) ph[u].w[e] = pack2(sacc[u][8 * t + 2 * e], sacc[u][8 * t + 2 * e + 1]);
        const int kpos = kb * 32 + 16 * t + 8 * g;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const Frag8 va = *reinterpret_cast<const Frag8*>(&vs[(c * 32 + lq) * VP + kpos]);
          o[0][c] = mfma32(va, ph[0], o[0][c]);
          o[1][c] = mfma32(va, ph[1], o[1][c]);
        }
      }
    }
  };

  dma(kbeg, ks0, vs0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kv0 = kbeg; kv0 < kend; kv0 += 2 * AK) {
    if (kv0 + AK < kend) dma(kv0 + AK, ks1, vs1);
    if (active) tile(kv0, ks0, vs0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kv0 + AK >= kend) break;
    if (kv0 + 2 * AK < kend) dma(kv0 + 2 * AK, ks0, vs0);
    if (active) tile(kv0 + AK, ks1, vs1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int qrow = qbase + 32 * u + lq;
    if (qrow >= p.sq) continue;
    // with ONES, element 8 of the last block is output row 32 (NC - 1) + 16 + 4 g: a ones row
    const float lsum = ONES ? o[u][NC - 1][8] : l_run[u];
    const float inv = 1.0f / lsum;
    bf16_t* out = out_row(b, h, qrow, m_run[u], lsum);
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + 8 * r4 + 4 * g;
        if (col >= D) continue;
        *reinterpret_cast<uint2*>(out + col) =
            make_uint2(pack2(o[u][c][4 * r4] * inv, o[u][c][4 * r4 + 1] * inv), pack2(o[u][c][4 * r4 + 2] * inv, o[u][c][4 * r4 + 3] * inv));
      }
  }
}

// Merge of the key ranges of attn_wide_kernel: thread (pair, query, 8 dims) weighs each range's
// normalised partial by exp2((m_r - max) scale) times its probability sum and divides by the
// weights' total; all ranges' loads are issued before any is used.
template <int D>
__global__ void __launch_bounds__(256) attn_merge_kernel(AttnArgs p) {
  constexpr int CH = D / 8;
  const int pairs = p.batch * p.n_q;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)pairs * p.sq * CH) return;
  const int ch = (int)(idx % CH);
  const long r = idx / CH;
  const int qrow = (int)(r % p.sq), pair = (int)(r / p.sq);
  const int h = pair % p.n_q, b = pair / p.n_q;
  const bf16_t* po = reinterpret_cast<const bf16_t*>(p.part);
  const float2* st = reinterpret_cast<const float2*>(po + (size_t)p.kv_parts * pairs * p.sq * D);
  const float scale = 1.4426950408889634f / sqrtf((float)D);
  float2 ml[3];
  Frag8 v[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const size_t row = ((size_t)min(k, p.kv_parts - 1) * pairs + pair) * p.sq + qrow;
    ml[k] = st[row];
    v[k] = *reinterpret_cast<const Frag8*>(po + row * D + 8 * ch);
  }
  float mx = ml[0].x;
#pragma unroll
  for (int k = 1; k < 3; ++k)
    if (k < p.kv_parts) mx = fmaxf(mx, ml[k].x);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, wsum = 0.f;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    if (k >= p.kv_parts) break;
    const float w = __builtin_amdgcn_exp2f((ml[k].x - mx) * scale) * ml[k].y;
    wsum += w;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += w * __uint_as_float(v[k].w[e] << 16);
      acc[2 * e + 1] += w * __uint_as_float(v[k].w[e] & 0xffff0000u);
    }
  }
  const float inv = 1.0f / wsum;
  Frag8 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o.w[e] = pack2(acc[2 * e] * inv, acc[2 * e + 1] * inv);
  *reinterpret_cast<Frag8*>(reinterpret_cast<bf16_t*>(p.out) + (size_t)b * p.o_batch + (size_t)qrow * p.o_row +
                            (size_t)h * D + 8 * ch) = o;
}

// Key ranges for the wide kernel: 2 or 3 when that fills the workgroup slots (2 per CU) at least
// 15 points better than one range (one 1008x1008 image: 336 workgroups leave a third of 512 slots
// empty; 3 ranges make 1008 of 1024), each range at least 8 tiles, and the scratch holds the
// partial rows.
static int wide_kv_parts(const AttnArgs& p, int D) {
  if (p.part == nullptr) return 1;
  const long wgs = (long)((p.sq + AQW - 1) / AQW) * p.n_q * p.batch;
  const long slots = 2L * (p.cus > 0 ? p.cus : 256);
  auto eff = [&](long u) { return (double)u / (double)(((u + slots - 1) / slots) * slots); };
  const int nkt = (p.sk + AK - 1) / AK;
  int best = 1;
  double best_eff = eff(wgs) + 0.15;
  for (int k = 2; k <= 3; ++k) {
    const size_t need = (size_t)k * p.batch * p.n_q * p.sq * (2 * D + 8);
    if (nkt < 8 * k || need > p.part_bytes) continue;
    if (eff(wgs * k) > best_eff + 1e-9) { best = k; best_eff = eff(wgs * k); }
  }
  return best;
}

// Key ranges of the causal kernel.  A causal query block of 128 reads every key up to its own
// last query, so the heaviest blocks take as many tiles as the sequence has, and on their own set
// the launch's length when all blocks run at once.  When the (pair, block) workgroups fit in one
// round of the GPU's workgroup slots (two per CU), the blocks are cut into ranges of at most tmax
// tiles, tmax the smallest (at least 4) that keeps the ranges within that one round, with at most
// 8 ranges per block and the fp32 partials within p.part.  A second round, or more partials,
// cost more than the shorter ranges save (the 1500-token prefill: attention 1.44 ms per pass
// unsplit, 1.09-1.13 ms in one round of ranges of 12 tiles, 1.16-1.21 ms with 10, 14 or 16 tiles,
// 1.38-1.45 ms with 4-8 tiles over two rounds; the 3579-token one, already past one round
// unsplit: 3.36-3.55 ms, 3.79 ms with only its 6 heaviest blocks per head cut in two, up to
// 5.2 ms cut finer: a cut block's merge lands on the end of the longest chain).
// Returns the ranges per pair (the grid is that times the pairs), or 0 when no block is cut
// (q.kv_tmax = 0).
template <int D>
static int causal_key_ranges(AttnArgs& q, int qblock, int threads) {
  q.kv_tmax = 0;
  if (q.part == nullptr || q.counters == nullptr || q.batch <= 0 || q.n_q <= 0) return 0;
  const int nqb = (q.sq + qblock - 1) / qblock, pairs = q.batch * q.n_q;
  const long slots_gpu = 2L * (q.cus > 0 ? q.cus : 256);
  if ((long)nqb * pairs > slots_gpu) return 0;
  auto tiles = [&](int qb) { return (std::min(q.sk, (qb + 1) * qblock) + AK - 1) / AK; };
  const int most = tiles(nqb - 1);
  constexpr size_t PV = (D + 31) / 32 * 16 + 2;        // fp32 values per thread and range
  for (int tmax = 4; tmax < most; ++tmax) {
    if ((most + tmax - 1) / tmax > 8) continue;
    int units = 0, slots = 0;
    for (int qb = 0; qb < nqb; ++qb) {
      const int P = (tiles(qb) + tmax - 1) / tmax;
      units += P;
      if (P > 1) slots += P;
    }
    if ((long)units * pairs > slots_gpu || (size_t)pairs * slots * PV * threads * sizeof(float) > q.part_bytes) continue;
    q.kv_tmax = tmax, q.kv_units = units, q.kv_slots = slots;
    return units;
  }
  return 0;
}

template <typename T, int D>
static hipError_t attn_launch(const AttnArgs& p, hipStream_t s) {
  if constexpr (sizeof(T) == 2 && D <= 80) {
    if (!p.causal) {
      AttnArgs q = p;
      q.kv_parts = wide_kv_parts(p, D);
      const int wgs = (p.sq + AQW - 1) / AQW * p.n_q * p.batch;
      hipLaunchKernelGGL((attn_wide_kernel<D>), dim3(wgs * q.kv_parts), dim3(256), 0, s, q);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess || q.kv_parts == 1) return e;
      const long n = (long)p.batch * p.n_q * p.sq * (D / 8);
      hipLaunchKernelGGL((attn_merge_kernel<D>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, q);
      return hipGetLastError();
    }
  }
  if (p.causal) {
    // 4 waves: workgroups of 2 waves (64 queries, twice as many, half as heavy) measured 60 us
    // against 51 us per layer on the 1500-token prefill (twice the K/V staging per query, and the
    // staging registers spill)
    constexpr int NW = 4;
    AttnArgs q = p;
    int units = causal_key_ranges<D>(q, NW * 32, NW * 64);
    if (units == 0) units = (p.sq + NW * 32 - 1) / (NW * 32);
    hipLaunchKernelGGL((attn_kernel<T, D, true, NW>), dim3(units * p.n_q * p.batch), dim3(NW * 64), 0, s, q);
  } else {
    hipLaunchKernelGGL((attn_kernel<T, D, false, 4>), dim3((p.sq + AQ - 1) / AQ * p.n_q * p.batch), dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

template <typename T>
hipError_t attention(const AttnArgs& p, int head_dim, hipStream_t s) {
  if (p.sq <= 0 || p.sk <= 0) return hipSuccess;
  if (p.n_kv <= 0 || p.n_q % p.n_kv || p.sk_pad % AK || p.sk_pad < p.sk) return hipErrorInvalidValue;
  switch (head_dim) {
    case 64: return attn_launch<T, 64>(p, s);
    case 80: return attn_launch<T, 80>(p, s);
    case 128:
      if constexpr (sizeof(T) == 2) return attn_launch<T, 128>(p, s);   // fp32 mode stops at d = 80
      break;
  }
  return hipErrorInvalidValue;
}

template hipError_t attention<bf16_t>(const AttnArgs&, int, hipStream_t);
template hipError_t attention<float>(const AttnArgs&, int, hipStream_t);

}  // namespace nova
