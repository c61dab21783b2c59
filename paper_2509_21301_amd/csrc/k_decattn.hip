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

template <typename T, int D>
__global__ void __launch_bounds__(256) dec_attn_kernel(DecAttnArgs p, int pairs_per_split) {
  constexpr bool F32 = sizeof(T) == 4;
  constexpr int NS = D / 32;      // k-steps of S = K Q^T
  constexpr int ND = D / 16;      // output row blocks of O^T
  __shared__ float sm_m[4][16], sm_l[4][16];
  __shared__ float sm_o[4][D][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int G = p.n_q / p.n_kv;
  const int col = lane & 15, grp = lane >> 4;
  const int ctx = p.pos[b] + 1;
  const int nblk = (ctx + DA_BLOCK - 1) / DA_BLOCK;
  const int pair_begin = split * pairs_per_split;
  const int pair_end = min(pair_begin + pairs_per_split, (nblk + 1) / 2);
  const T* kpool = reinterpret_cast<const T*>(p.kpool);
  const T* vpool = reinterpret_cast<const T*>(p.vpool);
  const int* table = p.tables + (size_t)b * p.max_blocks;

  // Q^T fragments: head col of this group, dims 32s + 8grp .. +8 (zero for col >= G)
  Frag8 qh[NS], ql[F32 ? NS : 1];
  const T* qsrc = reinterpret_cast<const T*>(p.q) + ((size_t)b * p.n_q + kvh * G + col) * D;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if (col < G) {
      if constexpr (F32) {
        float x[8];
        *reinterpret_cast<float4*>(x) = *reinterpret_cast<const float4*>(qsrc + 32 * s + 8 * grp);
        *reinterpret_cast<float4*>(x + 4) = *reinterpret_cast<const float4*>(qsrc + 32 * s + 8 * grp + 4);
        split8(x, qh[s], ql[s]);
      } else {
        qh[s] = *reinterpret_cast<const Frag8*>(qsrc + 32 * s + 8 * grp);
      }
    } else {
      qh[s] = zero_frag();
      if constexpr (F32) ql[s] = zero_frag();
    }
  }

  f32x4 o[ND];
#pragma unroll
  for (int i = 0; i < ND; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -1e30f, l_run = 0.f;
  const float scale = 1.4426950408889634f / sqrtf((float)D);

  for (int pr = pair_begin + wave; pr < pair_end; pr += 4) {
    f32x4 sc[2];
    int phys[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int blk = 2 * pr + j;
      phys[j] = blk < nblk ? table[blk] : -1;
      sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (phys[j] < 0) continue;
      const T* kb = kpool + ((size_t)phys[j] * p.n_kv + kvh) * DA_BLOCK * D;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const T* src = kb + (size_t)col * D + 32 * s + 8 * grp;     // token col, dims 32s+8grp..
        if constexpr (F32) {
          float x[8];
          *reinterpret_cast<float4*>(x) = *reinterpret_cast<const float4*>(src);
          *reinterpret_cast<float4*>(x + 4) = *reinterpret_cast<const float4*>(src + 4);
          Frag8 kh, kl;
          split8(x, kh, kl);
          sc[j] = mfma16(kh, qh[s], sc[j]);
          sc[j] = mfma16(kl, qh[s], sc[j]);
          sc[j] = mfma16(kh, ql[s], sc[j]);
        } else {
          Frag8 ka = *reinterpret_cast<const Frag8*>(src);
          sc[j] = mfma16(ka, qh[s], sc[j]);
        }
      }
    }
    // V^T fragments of both blocks, loaded now so that their latency overlaps the softmax: row
    // d = 16i + col, tokens 4grp..+3 of each block (zero past the table)
    uint2 vraw[ND][2];
    float4 vraw32[F32 ? ND : 1][2];
#pragma unroll
    for (int i = 0; i < ND; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const T* src = vpool + ((size_t)max(phys[j], 0) * p.n_kv + kvh) * D * DA_BLOCK + (size_t)(16 * i + col) * DA_BLOCK + 4 * grp;
        if constexpr (F32) {
          vraw32[i][j] = phys[j] >= 0 ? *reinterpret_cast<const float4*>(src) : float4{0.f, 0.f, 0.f, 0.f};
        } else {
          vraw[i][j] = phys[j] >= 0 ? *reinterpret_cast<const uint2*>(src) : make_uint2(0u, 0u);
        }
      }
    // lane holds S[token 4*grp + r][head col] for block j; mask tokens beyond the context
    float tmax = -1e30f;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int tok = (2 * pr + j) * DA_BLOCK + 4 * grp + r;
        const float v = (phys[j] >= 0 && tok < ctx) ? sc[j][r] * scale : -INFINITY;
        sc[j][r] = v;
        tmax = fmaxf(tmax, v);
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
      for (int r = 0; r < 4; ++r) {
        pv[4 * j + r] = exp2f(sc[j][r] - m_new);
        rs += pv[4 * j + r];
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
#pragma unroll
    for (int i = 0; i < ND; ++i) {
      o[i][0] *= corr; o[i][1] *= corr; o[i][2] *= corr; o[i][3] *= corr;
      // V^T fragment: row d = 16i + col, same tokens as the P^T fragment
      float vx[8];
      Frag8 va, vl;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if constexpr (F32) {
          *reinterpret_cast<float4*>(vx + 4 * j) = vraw32[i][j];
        } else {
          va.w[2 * j] = vraw[i][j].x; va.w[2 * j + 1] = vraw[i][j].y;
        }
      }
      if constexpr (F32) {
        split8(vx, va, vl);
        o[i] = mfma16(va, ph, o[i]);
        o[i] = mfma16(vl, ph, o[i]);
        o[i] = mfma16(va, pl, o[i]);
      } else {
        o[i] = mfma16(va, ph, o[i]);
      }
    }
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

// Log-sum-exp combine of the context splits: one workgroup of D threads per (sequence, head);
// split statistics are read in parallel, then every thread sums its dimension over the splits.
template <typename T, int D>
__global__ void __launch_bounds__(D) dec_attn_combine(DecAttnArgs p, int nsplit) {
  __shared__ float wts[64];
  __shared__ float norm;
  const int bh = blockIdx.x;                 // b * n_q + head
  const float* part = p.partial + (size_t)bh * nsplit * (D + 2);
  const int t = threadIdx.x;
  float m = -1e30f;
  if (t < nsplit) m = part[t * (D + 2)];
  float M = wave_max(t < 64 ? m : -1e30f);
  if (t < 64) {
    const float w = t < nsplit ? exp2f(m - M) : 0.f;
    const float lw = wave_sum(t < nsplit ? w * part[t * (D + 2) + 1] : 0.f);
    wts[t] = w;
    if (t == 0) norm = 1.0f / lw;
  }
  __syncthreads();
  float O = 0.f;
  for (int sp = 0; sp < nsplit; ++sp) O += wts[sp] * part[sp * (D + 2) + 2 + t];
  reinterpret_cast<T*>(p.out)[(size_t)bh * D + t] = from_f<T>(O * norm);
}

template <typename T, int D>
static hipError_t dec_launch(const DecAttnArgs& p, hipStream_t s) {
  const int nsplit = dec_splits(p.B, p.n_kv, p.max_ctx);
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
  if (p.block != DA_BLOCK || p.n_kv <= 0 || p.n_q % p.n_kv || p.n_q / p.n_kv > 16 || p.max_ctx <= 0)
    return hipErrorInvalidValue;
  switch (head_dim) {
    case 64: return dec_launch<T, 64>(p, s);
    case 128: return dec_launch<T, 128>(p, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t decode_attention<bf16_t>(const DecAttnArgs&, int, hipStream_t);
template hipError_t decode_attention<float>(const DecAttnArgs&, int, hipStream_t);

}  // namespace nova
