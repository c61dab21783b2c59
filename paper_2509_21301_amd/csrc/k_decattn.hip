// Paged decode attention: each sequence's single query attends to its cached keys/values,
// which live in fixed 16-token blocks addressed through a block table (PagedAttention-style
// cache, the paper's Sec. 1 and Sec. 5.1).  Decode is memory-bound (the paper's Table 3), so
// the kernel is shaped to stream the KV blocks at HBM rate:
//  * grid = (context splits, KV heads, sequences); a wave takes pairs of blocks (32 tokens);
//  * the G query heads sharing a KV head form the 16-wide MFMA operand, so K and V are read
//    once per group: S = K Q^T (16 tokens x 16 heads per MFMA 16x16x32) and
//    O^T = V^T P^T (V blocks are stored transposed, [d][16 tokens], so the contraction over
//    tokens reads 8 contiguous bytes per lane);
//  * the per-head max and sum over tokens are wavefront shuffles (lane ^ 16, lane ^ 32);
//    waves are merged through LDS and splits by a second pass (log-sum-exp combine).
// The step's own token is folded in: the kernel sums the QKV projection's split-K slabs, applies
// the rotary embedding to q and k (the sines and cosines of the sequence's position come from a
// table the step computes once for all layers), and the wave whose block pair holds that
// position appends k and v to the cache and uses them in place of the slot's old contents.
// So no rotary/append pass runs between the QKV projection and the attention.
// K pool layout: [num_blocks][n_kv][16][D];  V pool layout: [num_blocks][n_kv][D][16].
#include "common.hpp"
#include "kernels.hpp"

namespace nova {

constexpr int DA_BLOCK = 16;
constexpr int DA_TOK_PER_SPLIT_MIN = 128;

static int dec_splits(int B, int n_kv, int max_ctx) {
  const int pairs = (max_ctx + 31) / 32;
  const int want = (512 + B * n_kv - 1) / (B * n_kv);
  int per = (pairs + want - 1) / want;                  // block pairs per split
  per = max(per, DA_TOK_PER_SPLIT_MIN / 32);
  int n = (pairs + per - 1) / per;
  while (n > 64) n = (pairs + ++per - 1) / per;      // the combine holds at most 64 splits
  return n;
}

size_t dec_attn_partial_floats(int B, int n_q, int D, int max_ctx, int n_kv) {
  const int s = dec_splits(B, n_kv, max_ctx);
  return (size_t)B * n_q * s * (D + 2);
}

// Raw registers of one block pair: K rows (token col, 8 dims per 32-dim step) and V^T rows
// (dim 16i + col, tokens 4grp..+3) of both blocks, with the blocks' physical ids (-1: none).
template <bool F32, int NS, int ND> struct DaPair;
template <int NS, int ND> struct DaPair<false, NS, ND> { Frag8 k[2][NS]; uint2 v[ND][2]; int ph[2]; };
template <int NS, int ND> struct DaPair<true, NS, ND> { float4 k[2][NS][2]; float4 v[ND][2]; int ph[2]; };

template <typename T, int D>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) dec_attn_kernel(DecAttnArgs p, int pairs_per_split) {
  constexpr bool F32 = sizeof(T) == 4;
  constexpr int NS = D / 32;      // k-steps of S = K Q^T
  constexpr int ND = D / 16;      // output row blocks of O^T
  using Pair = DaPair<F32, NS, ND>;
  constexpr int HALF = D / 2;
  __shared__ float sm_m[4][16], sm_l[4][16];
  __shared__ float sm_o[4][D][16];
  __shared__ __align__(16) T sm_q[16][D];        // the step's rotated q of the group's heads
  __shared__ __align__(16) T sm_nk[D];           // the new token's rotated k and its v
  __shared__ T sm_nv[D];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int G = p.n_q / p.n_kv;
  const int col = lane & 15, grp = lane >> 4;
  // a position past the documented bound (pos + 1 <= max_ctx, which the block-table width covers)
  // is clamped, so no table or cache access leaves the sequence's row whatever the caller passes
  const int ps = min(max(p.pos[b], 0), p.max_ctx - 1);
  const int ctx = ps + 1;
  const int nblk = (ctx + DA_BLOCK - 1) / DA_BLOCK;
  const int pair_begin = split * pairs_per_split;
  const int pair_end = min(pair_begin + pairs_per_split, (nblk + 1) / 2);
  const T* kpool = reinterpret_cast<const T*>(p.kpool);
  const T* vpool = reinterpret_cast<const T*>(p.vpool);
  const int* table = p.tables + (size_t)b * p.max_blocks;
  // this wave takes pairs first, first + 4, ...: iteration it covers pair first + 4 it
  const int first = pair_begin + wave;
  const int n_it = first < pair_end ? (pair_end - first + 3) / 4 : 0;
  // the new token (position ps) is slot ps % 16 of block ps / 16, in the context's last pair;
  // it_new: this wave's iteration over that pair (-1: another wave's)
  const int new_blk = ps / DA_BLOCK, slot = ps % DA_BLOCK;
  const int new_pair = new_blk / 2, jn = new_blk & 1;
  const int it_new = new_pair >= first && new_pair < pair_end && ((new_pair - first) & 3) == 0 ? (new_pair - first) >> 2 : -1;

  // block-table entries of 32 iterations at a time, one per lane (lane 2i + j: block j of
  // iteration i), read back with a uniform lane index, so the K/V loads of a pair wait for no
  // table load of their own
  int tl = -1, tl_chunk = -1;
  auto phys_of = [&](int it, int j) -> int {
    if ((it >> 5) != tl_chunk) {
      tl_chunk = it >> 5;
      const int pr = first + 4 * (32 * tl_chunk + (lane >> 1));
      const int blk = 2 * pr + (lane & 1);
      tl = (pr < pair_end && blk < nblk) ? table[blk] : -1;
    }
    return __builtin_amdgcn_readlane(tl, 2 * (it & 31) + j);
  };
  // every load of a pair is issued together (addresses clamped to block 0 where a block is absent)
  auto load = [&](int it, Pair& r) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      r.ph[j] = phys_of(it, j);
      const size_t base = ((size_t)max(r.ph[j], 0) * p.n_kv + kvh) * DA_BLOCK * D;
      const T* kb = kpool + base + (size_t)col * D + 8 * grp;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        if constexpr (F32) {
          r.k[j][s][0] = *reinterpret_cast<const float4*>(kb + 32 * s);
          r.k[j][s][1] = *reinterpret_cast<const float4*>(kb + 32 * s + 4);
        } else {
          r.k[j][s] = *reinterpret_cast<const Frag8*>(kb + 32 * s);
        }
      }
      const T* vb = vpool + base + (size_t)col * DA_BLOCK + 4 * grp;
#pragma unroll
      for (int i = 0; i < ND; ++i) {
        if constexpr (F32) r.v[i][j] = *reinterpret_cast<const float4*>(vb + (size_t)16 * i * DA_BLOCK);
        else r.v[i][j] = *reinterpret_cast<const uint2*>(vb + (size_t)16 * i * DA_BLOCK);
      }
    }
  };

  // two register sets: the loads of the next pair are in flight while this pair is computed
  Pair ra, rb;
  if (n_it > 0) load(0, ra);

  // The step's q for the G heads of this group and, in the workgroup whose splits hold the new
  // token, its k and v: the projection's split-K slabs summed in order, q and k rotated (dim c <
  // D/2 pairs with c + D/2), staged in LDS in the activation type.  Every load is requested before
  // any is summed (4 slabs at a time), so this costs one round trip to memory, taken while the
  // first K/V loads are in flight.  Thread t takes rotation pairs t, t + 256, ... (head h = pair /
  // (D/2), h == G: the new k) and, when t < D, dimension t of the new v.
  const bool owner_wg = new_pair >= pair_begin && new_pair < pair_end;
  {
    constexpr int PPT = (17 * HALF + 255) / 256;      // pairs per thread at most (G <= 16, plus k)
    const int npairs = (G + (owner_wg ? 1 : 0)) * HALF;
    const size_t qkvw = (size_t)(p.n_q + 2 * p.n_kv) * D;
    int off[PPT];
    float sn[PPT], cs[PPT], a1[PPT], a2[PPT], av = 0.f;
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
      const int pi = min(tid + 256 * u, npairs - 1);        // clamped: the duplicates are not stored
      const int h = pi / HALF, c = pi % HALF;
      off[u] = (h < G ? kvh * G + h : p.n_q + kvh) * D + c;
      sn[u] = p.rope[(size_t)b * D + c];
      cs[u] = p.rope[(size_t)b * D + HALF + c];
      a1[u] = a2[u] = 0.f;
    }
    const int voff = (p.n_q + p.n_kv + kvh) * D + (tid % D);
    for (int sp0 = 0; sp0 < p.qkv_splits; sp0 += 4) {
      float t1[4][PPT], t2[4][PPT], tv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float* r = p.qkv + ((size_t)min(sp0 + q, p.qkv_splits - 1) * p.B + b) * qkvw;
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
          t1[q][u] = r[off[u]];
          t2[q][u] = r[off[u] + HALF];
        }
        tv[q] = r[voff];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (sp0 + q < p.qkv_splits) {
#pragma unroll
          for (int u = 0; u < PPT; ++u) { a1[u] += t1[q][u]; a2[u] += t2[q][u]; }
          av += tv[q];
        }
    }
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
      const int pi = tid + 256 * u;
      if (pi >= npairs) break;
      const int h = pi / HALF, c = pi % HALF;
      const float y1 = a1[u] * cs[u] - a2[u] * sn[u], y2 = a2[u] * cs[u] + a1[u] * sn[u];
      T* dst = h < G ? sm_q[h] : sm_nk;
      dst[c] = from_f<T>(y1);
      dst[c + HALF] = from_f<T>(y2);
    }
    if (owner_wg && tid < D) sm_nv[tid] = from_f<T>(av);
  }
  __syncthreads();

  // Q^T fragments: head col of this group, dims 32s + 8grp .. +8 (zero for col >= G)
  Frag8 qh[NS], ql[F32 ? NS : 1];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if (col < G) {
      const T* qs = sm_q[col] + 32 * s + 8 * grp;
      if constexpr (F32) {
        float x[8];
        *reinterpret_cast<float4*>(x) = *reinterpret_cast<const float4*>(qs);
        *reinterpret_cast<float4*>(x + 4) = *reinterpret_cast<const float4*>(qs + 4);
        split8(x, qh[s], ql[s]);
      } else {
        qh[s] = *reinterpret_cast<const Frag8*>(qs);
      }
    } else {
      qh[s] = zero_frag();
      if constexpr (F32) ql[s] = zero_frag();
    }
  }
  // the new token appended to the cache (K row, V^T column)
  if (owner_wg && tid < D) {
    const size_t base = ((size_t)table[new_blk] * p.n_kv + kvh) * DA_BLOCK * D;
    const_cast<T*>(kpool)[base + (size_t)slot * D + tid] = sm_nk[tid];
    const_cast<T*>(vpool)[base + (size_t)tid * DA_BLOCK + slot] = sm_nv[tid];
  }
  // the owner wave's registers of block jn take the new token, whatever the cache held there
  // (jn and slot are uniform: the branches select registers, they do not index them)
  auto patch = [&](Pair& r) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (j != jn) continue;
      if (col == slot) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          if constexpr (F32) {
            r.k[j][s][0] = *reinterpret_cast<const float4*>(sm_nk + 32 * s + 8 * grp);
            r.k[j][s][1] = *reinterpret_cast<const float4*>(sm_nk + 32 * s + 8 * grp + 4);
          } else {
            r.k[j][s] = *reinterpret_cast<const Frag8*>(sm_nk + 32 * s + 8 * grp);
          }
        }
      }
      if (grp == slot / 4) {
        const int e = slot & 3;
#pragma unroll
        for (int i = 0; i < ND; ++i) {
          const T v = sm_nv[16 * i + col];
          if constexpr (F32) {
            if (e == 0) r.v[i][j].x = v;
            else if (e == 1) r.v[i][j].y = v;
            else if (e == 2) r.v[i][j].z = v;
            else r.v[i][j].w = v;
          } else {
            const uint32_t keep = (e & 1) ? 0x0000ffffu : 0xffff0000u;
            const uint32_t put = (uint32_t)v << (16 * (e & 1));
            if (e < 2) r.v[i][j].x = (r.v[i][j].x & keep) | put;
            else r.v[i][j].y = (r.v[i][j].y & keep) | put;
          }
        }
      }
    }
  };

  f32x4 o[ND];
#pragma unroll
  for (int i = 0; i < ND; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -1e30f, l_run = 0.f;
  const float scale = 1.4426950408889634f / sqrtf((float)D);

  auto compute = [&](int it, const Pair& r) {
    const int pr = first + 4 * it;
    f32x4 sc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        if constexpr (F32) {
          float x[8];
          *reinterpret_cast<float4*>(x) = r.k[j][s][0];
          *reinterpret_cast<float4*>(x + 4) = r.k[j][s][1];
          Frag8 kh, kl;
          split8(x, kh, kl);
          sc[j] = mfma16(kh, qh[s], sc[j]);
          sc[j] = mfma16(kl, qh[s], sc[j]);
          sc[j] = mfma16(kh, ql[s], sc[j]);
        } else {
          sc[j] = mfma16(r.k[j][s], qh[s], sc[j]);
        }
      }
    }
    // lane holds S[token 4*grp + q][head col] for block j; mask tokens beyond the context (and
    // absent blocks: the K rows read there are block 0's, replaced by -inf here)
    float tmax = -1e30f;
    int nvalid[2];       // tokens 4grp..+3 of block j inside the context
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int t0 = (2 * pr + j) * DA_BLOCK + 4 * grp;
      nvalid[j] = r.ph[j] < 0 ? 0 : min(max(ctx - t0, 0), 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float v = q < nvalid[j] ? sc[j][q] * scale : -INFINITY;
        sc[j][q] = v;
        tmax = fmaxf(tmax, v);
      }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float corr = exp2f(m_run - m_new);
    float rs = 0.f;
    float pv[8];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        pv[4 * j + q] = exp2f(sc[j][q] - m_new);
        rs += pv[4 * j + q];
      }
    rs += __shfl_xor(rs, 16, 64);
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * corr + rs;
    m_run = m_new;
    // P^T fragment: head col, tokens (block 0: 4grp..+3, block 1: 4grp..+3)
    Frag8 ph, pl;
    if constexpr (F32) split8(pv, ph, pl);
    else {
#pragma unroll
      for (int e = 0; e < 4; ++e) ph.w[e] = pack2(pv[2 * e], pv[2 * e + 1]);
    }
    // V^T values of tokens outside the context are zeroed (their probabilities are zero, but the
    // cache slots past the last written token may hold anything, NaN included)
    uint32_t vmask[2][2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const unsigned long long m = nvalid[j] >= 4 ? ~0ull : ((1ull << (16 * nvalid[j])) - 1ull);
      vmask[j][0] = (uint32_t)m;
      vmask[j][1] = (uint32_t)(m >> 32);
    }
#pragma unroll
    for (int i = 0; i < ND; ++i) {
      o[i][0] *= corr; o[i][1] *= corr; o[i][2] *= corr; o[i][3] *= corr;
      // V^T fragment: row d = 16i + col, same tokens as the P^T fragment
      if constexpr (F32) {
        float vx[8];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          vx[4 * j + 0] = nvalid[j] > 0 ? r.v[i][j].x : 0.f;
          vx[4 * j + 1] = nvalid[j] > 1 ? r.v[i][j].y : 0.f;
          vx[4 * j + 2] = nvalid[j] > 2 ? r.v[i][j].z : 0.f;
          vx[4 * j + 3] = nvalid[j] > 3 ? r.v[i][j].w : 0.f;
        }
        Frag8 va, vl;
        split8(vx, va, vl);
        o[i] = mfma16(va, ph, o[i]);
        o[i] = mfma16(vl, ph, o[i]);
        o[i] = mfma16(va, pl, o[i]);
      } else {
        Frag8 va;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          va.w[2 * j] = r.v[i][j].x & vmask[j][0];
          va.w[2 * j + 1] = r.v[i][j].y & vmask[j][1];
        }
        o[i] = mfma16(va, ph, o[i]);
      }
    }
  };

  for (int it = 0; it < n_it; it += 2) {
    if (it + 1 < n_it) load(it + 1, rb);
    if (it == it_new) patch(ra);
    compute(it, ra);
    if (it + 1 >= n_it) break;
    if (it + 2 < n_it) load(it + 2, ra);
    if (it + 1 == it_new) patch(rb);
    compute(it + 1, rb);
  }

  // merge the four waves: lane holds O^T[d = 16i + 4grp + r][head col]
  if (grp == 0) { sm_m[wave][col] = m_run; sm_l[wave][col] = l_run; }
#pragma unroll
  for (int i = 0; i < ND; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) sm_o[wave][16 * i + 4 * grp + r][col] = o[i][r];
  __syncthreads();
  const int nsplit = gridDim.x;
  for (int idx = tid; idx < G * D; idx += 256) {
    const int hh = idx / D, d = idx % D;
    float M = -1e30f;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, sm_m[w][hh]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = exp2f(sm_m[w][hh] - M);
      L += f * sm_l[w][hh];
      O += f * sm_o[w][d][hh];
    }
    const int head = kvh * G + hh;
    if (nsplit == 1) {
      reinterpret_cast<T*>(p.out)[((size_t)b * p.n_q + head) * D + d] = from_f<T>(O / L);
    } else {
      float* part = p.partial + (((size_t)b * p.n_q + head) * nsplit + split) * (D + 2);
      part[2 + d] = O;
      if (d == 0) { part[0] = M; part[1] = L; }
    }
  }
}

// Log-sum-exp combine of the context splits: one workgroup of D threads per (sequence, head).
// Every load is issued before any is used (the first 16 splits' outputs of the thread's dimension,
// and in wave 0 each split's max and sum), so the kernel waits for one round trip to memory
// rather than three; every thread then sums its dimension over the splits in split order.
template <typename T, int D>
__global__ void __launch_bounds__(D) dec_attn_combine(DecAttnArgs p, int nsplit) {
  constexpr int PF = 16;
  __shared__ float wts[64];
  __shared__ float norm;
  const int bh = blockIdx.x;                 // b * n_q + head
  const float* part = p.partial + (size_t)bh * nsplit * (D + 2);
  const int t = threadIdx.x;
  float ov[PF];
#pragma unroll
  for (int sp = 0; sp < PF; ++sp) ov[sp] = sp < nsplit ? part[sp * (D + 2) + 2 + t] : 0.f;
  float m = -1e30f, l = 0.f;
  if (t < nsplit) {
    m = part[t * (D + 2)];
    l = part[t * (D + 2) + 1];
  }
  float M = wave_max(t < 64 ? m : -1e30f);
  if (t < 64) {
    const float w = t < nsplit ? exp2f(m - M) : 0.f;
    const float lw = wave_sum(t < nsplit ? w * l : 0.f);
    wts[t] = w;
    if (t == 0) norm = 1.0f / lw;
  }
  __syncthreads();
  float O = 0.f;
#pragma unroll
  for (int sp = 0; sp < PF; ++sp)
    if (sp < nsplit) O += wts[sp] * ov[sp];
  for (int sp = PF; sp < nsplit; ++sp) O += wts[sp] * part[sp * (D + 2) + 2 + t];
  reinterpret_cast<T*>(p.out)[(size_t)bh * D + t] = from_f<T>(O * norm);
}

template <typename T, int D>
static hipError_t dec_launch(const DecAttnArgs& p, hipStream_t s) {
  const int nsplit = dec_splits(p.B, p.n_kv, p.max_ctx);
  if (nsplit > 1 && p.partial == nullptr) return hipErrorInvalidValue;
  const int pairs = (p.max_ctx + 31) / 32;
  const int per = (pairs + nsplit - 1) / nsplit;
  hipLaunchKernelGGL((dec_attn_kernel<T, D>), dim3(nsplit, p.n_kv, p.B), dim3(256), 0, s, p, per);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nsplit == 1) return e;
  hipLaunchKernelGGL((dec_attn_combine<T, D>), dim3(p.B * p.n_q), dim3(D), 0, s, p, nsplit);
  return hipGetLastError();
}

template <typename T>
hipError_t decode_attention(const DecAttnArgs& p, int head_dim, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.block != DA_BLOCK || p.n_kv <= 0 || p.n_q % p.n_kv || p.n_q / p.n_kv > 16 || p.max_ctx <= 0 ||
      p.qkv == nullptr || p.qkv_splits <= 0)
    return hipErrorInvalidValue;
  switch (head_dim) {
    case 64: return dec_launch<T, 64>(p, s);
    case 128:
      if constexpr (sizeof(T) == 4) return hipErrorInvalidValue;   // the fp32 mode stops at head_dim 80
      else return dec_launch<T, 128>(p, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t decode_attention<bf16_t>(const DecAttnArgs&, int, hipStream_t);
template hipError_t decode_attention<float>(const DecAttnArgs&, int, hipStream_t);

}  // namespace nova
