// Multi-hop relevance (App. A.4 eq:app_global_seed_score,
// eq:app_hop_propagation, eq:app_diffused_relevance, eq:app_bottom_up_value).
//
// Runs inside gracekv_build_trees when lambda_graph > 0, once the relevance
// row statistics (m_V, Z_V per window query) and the per-(l, g) sums S_{l,g}
// are known:
//   * s-hat of every (l, g) is in the token-value array: bf16 caches from the
//     token relevance pass below (run for every build; the root kernel later
//     overwrites the values with the mix); fp32 caches from a first run of the
//     root kernel;
//   * k_mh_seed_score: S_t = mean over (l, g) of s-hat_{l,g,t};
//   * k_mh_top + k_mh_seeds: the positions in descending score (ties to the
//     smaller position) while their cumulative share of the total stays below
//     0.9 (the one reaching it included), at most 64, weights proportional to
//     the score.  k_mh_top keeps the 64 largest keys of each 4096-token block,
//     k_mh_seeds (one workgroup) takes the seeds from those candidates;
//   * two passes per hop over (propagation layer, KV head, token chunk):
//     pass 0 gives each seed row's maximum and partition sum over its causal
//     range [0, u]; pass 1 sums w_u pi_{u,t} over the rows for every token;
//   * k_mh_hop_reduce: d^(k)_t over layers and heads, zero at the current and
//     earlier seeds, accumulated with the decay 0.5^(k-1);
//   * k_mh_finish: d-hat = d / (sum_C d + eps).
// The root kernel then mixes R^tok = (1 - lambda) s-hat + lambda d-hat.
//
// Row layout: a group is (propagation layer, KV head) for the hops and (layer,
// KV head) for the direct pass; row j of query head slot hl is r = 64 hl + j,
// j a seed (hops) or a window query (direct pass).  bf16 caches run the logits
// on MFMA (16x16x32: 16 tokens x 16 rows per tile, the bf16 products exact in
// fp32, summed in fp32 like the reference dot product), one wave per query
// head slot, 64-token blocks of keys staged in LDS.  fp32 caches use one
// thread per row on the vector ALUs.
#include "common.h"

namespace gkv {

constexpr int MH_SEEDS = 64;                 // at most this many seeds per hop
constexpr int MH_HOPS = 2;
constexpr int MH_CH = 1024;                  // tokens per workgroup of the row passes
constexpr int MH_SUB = 64;                   // tokens staged at once
constexpr int MH_PF = 4;                     // staging rounds prefetched into registers
constexpr int MH_TOPB = 4096;                // tokens per block of the candidate pass
constexpr double MH_ETA = 0.9;               // cumulative seed share
constexpr float MH_RHO = 0.5f;               // inter-hop decay
constexpr float LOG2E = 1.44269504088896341f;

static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

MhView mh_view(void* base, const Dims& dm) {
  // offsets first (base may be null when only the size is wanted)
  const size_t N = (size_t)dm.N_c;
  const int rmax = dm.hpg * MH_SEEDS;
  const int ngrp = dm.n_gl * dm.G;
  const int nz = (rmax + 255) / 256;
  const int nch = (int)((N + MH_CH - 1) / MH_CH);
  const size_t ntop = (N + MH_TOPB - 1) / MH_TOPB;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o += al(bytes); return at; };
  const size_t o_dk = take(N * 4), o_dacc = take(N * 4), o_dhat = take(N * 4);
  const size_t o_seeds = take(MH_SEEDS * 4), o_wts = take(MH_SEEDS * 4), o_ns = take(16);
  const size_t o_used = take(MH_HOPS * MH_SEEDS * 4), o_nused = take(16);
  const size_t o_rstat = take((size_t)ngrp * rmax * 8), o_rpart = take((size_t)nch * ngrp * rmax * 8);
  const size_t o_dpart = take((size_t)ngrp * nz * N * 4);
  const size_t o_cand = take(ntop * MH_SEEDS * 8), o_bsum = take(ntop * 8);
  MhView v{};
  v.bytes = o;
  if (base) {
    char* b = (char*)base;
    v.dk = (float*)(b + o_dk); v.dacc = (float*)(b + o_dacc); v.dhat = (float*)(b + o_dhat);
    v.seeds = (int32_t*)(b + o_seeds); v.wts = (float*)(b + o_wts); v.ns = (int32_t*)(b + o_ns);
    v.used = (int32_t*)(b + o_used); v.nused = (int32_t*)(b + o_nused);
    v.rstat = (float2*)(b + o_rstat); v.rpart = (float2*)(b + o_rpart); v.dpart = (float*)(b + o_dpart);
    v.cand = (uint64_t*)(b + o_cand); v.bsum = (double*)(b + o_bsum);
  }
  return v;
}

size_t mh_bytes(const Dims& dm) { return dm.lam_graph > 0.f ? mh_view(nullptr, dm).bytes : 0; }

__global__ void k_mh_seed_score(Dims dm, TreeView tv, MhView mh) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= dm.N_c) return;
  const int64_t LG = (int64_t)dm.L * dm.G;
  double s = 0.0;
  for (int64_t lg = 0; lg < LG; ++lg) s += tv.tok_R[lg * dm.N_c + t];
  mh.dk[t] = (float)(s / (double)LG);
  if (t == 0) *mh.nused = 0;
}

// (score, -position) as one ordered key; scores are >= 0
__device__ __forceinline__ uint64_t mh_key(float s, int64_t t) {
  return ((uint64_t)__float_as_uint(s > 0.f ? s : 0.f) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)t);
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t b = __shfl_xor(v, o, 64);
    v = b > v ? b : v;
  }
  return v;
}

// The 64 largest keys of one block of MH_TOPB scores (descending, 0 past the
// block's size) and the block's score sum.
__global__ __launch_bounds__(256) void k_mh_top(Dims dm, MhView mh) {
  __shared__ float ss[MH_TOPB];
  __shared__ unsigned long long skey[4];
  __shared__ double sred[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t b0 = (int64_t)blockIdx.x * MH_TOPB;
  const int n = (int)(dm.N_c - b0 < MH_TOPB ? dm.N_c - b0 : MH_TOPB);
  double a = 0.0;
  for (int i = tid; i < n; i += 256) {
    const float v = mh.dk[b0 + i];
    ss[i] = v;
    a += v;
  }
  a = wave_sum(a);
  if (lane == 0) sred[wave] = a;
  __syncthreads();
  if (tid == 0) mh.bsum[blockIdx.x] = (sred[0] + sred[1]) + (sred[2] + sred[3]);
  uint64_t prev = ~0ull;
  for (int k = 0; k < MH_SEEDS; ++k) {
    uint64_t best = 0;
    for (int i = tid; i < n; i += 256) {
      const uint64_t key = mh_key(ss[i], b0 + i);
      if (key < prev && key > best) best = key;
    }
    best = wave_max_u64(best);
    if (lane == 0) skey[wave] = best;
    __syncthreads();
    uint64_t b = skey[0];
    for (int w = 1; w < 4; ++w) b = skey[w] > b ? skey[w] : b;
    __syncthreads();
    if (tid == 0) mh.cand[(int64_t)blockIdx.x * MH_SEEDS + k] = b;
    prev = b;
  }
}

// Seeds from the block candidates: every key among the 64 largest overall is
// among its block's 64 largest.
__global__ __launch_bounds__(1024) void k_mh_seeds(Dims dm, MhView mh) {
  __shared__ double sred[16];
  __shared__ unsigned long long skey[16];
  __shared__ float swt[MH_SEEDS];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nb = (int)((dm.N_c + MH_TOPB - 1) / MH_TOPB);
  const int nc = nb * MH_SEEDS;
  double a = 0.0;
  for (int b = tid; b < nb; b += 1024) a += mh.bsum[b];
  a = wave_sum(a);
  if (lane == 0) sred[wave] = a;
  __syncthreads();
  double total = 0.0;
  for (int w = 0; w < 16; ++w) total += sred[w];
  const int nused0 = *mh.nused;
  uint64_t prev = ~0ull;
  double cum = 0.0, wsum = 0.0;
  int ns = 0;
  for (int k = 0; k < MH_SEEDS; ++k) {
    if (!(total > 0.0) || cum >= MH_ETA) break;
    uint64_t best = 0;
    for (int i = tid; i < nc; i += 1024) {
      const uint64_t key = mh.cand[i];
      if (key < prev && key > best) best = key;
    }
    best = wave_max_u64(best);
    if (lane == 0) skey[wave] = best;
    __syncthreads();
    uint64_t b = skey[0];
    for (int w = 1; w < 16; ++w) b = skey[w] > b ? skey[w] : b;
    __syncthreads();
    const float s = __uint_as_float((uint32_t)(b >> 32));
    if (!(s > 0.f)) break;
    const int t = (int)(0xFFFFFFFFu - (uint32_t)(b & 0xFFFFFFFFu));
    if (tid == 0) { mh.seeds[ns] = t; swt[ns] = s; mh.used[nused0 + ns] = t; }
    cum += (double)s / total;
    wsum += (double)s;
    ++ns;
    prev = b;
  }
  __syncthreads();
  if (tid < ns) mh.wts[tid] = (float)((double)swt[tid] / wsum);
  if (tid == 0) { *mh.ns = ns; *mh.nused = nused0 + ns; }
}

// ---------------------------------------------------------------------------
// bf16: relevance rows on MFMA.  RR_HOP_STATS: hop row statistics;
// RR_HOP_SUMS: hop token sums; RR_DIRECT: direct relevance s-hat of (l, g) into
// the token values (the token relevance pass).  Block:
// one wave per query head slot of the group (hpg waves).
// ---------------------------------------------------------------------------
enum { RR_HOP_STATS = 0, RR_HOP_SUMS = 1, RR_DIRECT = 2 };

template <int D, int MODE>
__global__ __launch_bounds__(512) void k_rel_rows(Dims dm, const uint16_t* __restrict__ K,
                                                 const uint16_t* __restrict__ Qs, TreeView tv, MhView mh) {
  constexpr int KS = D / 32;
  constexpr int LDK = D + 8;                  // staged key row stride (bf16): conflict-free fragment reads
  constexpr int C8 = D / 8;                   // 16-byte chunks per key row
  __shared__ __align__(16) uint16_t sk[MH_SUB * LDK];
  __shared__ float red[8][MH_SUB];
  const int ch = blockIdx.x, grp = blockIdx.y;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
  const int nw = blockDim.x >> 6;
  const int gi = MODE == RR_DIRECT ? 0 : grp / dm.G;
  const int g = grp % dm.G;
  const int l = MODE == RR_DIRECT ? grp / dm.G : dm.gl[gi];
  const int h = g * dm.hpg + w;               // the wave's query head
  const int nrow = MODE == RR_DIRECT ? dm.W : *mh.ns;
  const int rmax = dm.hpg * MH_SEEDS;
  const float sc2 = LOG2E / sqrtf((float)D);
  // the wave's rows j = 16 rt + i16: query fragment, causal limit, weight, log2 normaliser
  uint4 qf[4][KS];
  int uj[4];
  float wj[4], cj[4];
  int umax = -1;
  if (MODE != RR_DIRECT)
    for (int s = 0; s < nrow; ++s) umax = max(umax, mh.seeds[s]);
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    const int j = 16 * rt + i16;
    const bool ok = j < nrow;
    const uint16_t* qrow;
    if (MODE == RR_DIRECT) {
      qrow = Qs + (((int64_t)l * dm.H + h) * dm.W + (ok ? j : 0)) * D;
      uj[rt] = ok ? 0x7fffffff : -1;
      wj[rt] = ok ? 1.f : 0.f;
      cj[rt] = INFINITY;                      // a masked row (zero query) contributes 2^(-inf) = 0
      if (ok) {
        const float4 st = tv.row_stats[((int64_t)l * dm.G + g) * dm.rows + w * dm.W + j];
        cj[rt] = st.x * LOG2E + __log2f(st.y);
      }
    } else {
      const int u = ok ? mh.seeds[j] : 0;
      qrow = Qs + (((int64_t)gi * dm.H + h) * dm.T + u) * D;
      uj[rt] = ok ? u : -1;
      wj[rt] = ok ? mh.wts[j] : 0.f;
      cj[rt] = 0.f;
      if (MODE == RR_HOP_SUMS && ok) {
        const float2 st = mh.rstat[(int64_t)grp * rmax + w * MH_SEEDS + j];
        cj[rt] = st.x + st.y;
      }
    }
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qf[rt][s] = ok ? *(const uint4*)(qrow + 32 * s + 8 * g4) : make_uint4(0, 0, 0, 0);
  }
  // direct pass: the normaliser of row 16 rt + 4 g4 + r, the lane's rows once
  // the products are taken with the rows as M and the tokens as N (+inf for a
  // row past the last: 2^(-inf) = 0)
  float cT[4][4];
  if (MODE == RR_DIRECT) {
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = 16 * rt + 4 * g4 + r;
        cT[rt][r] = INFINITY;
        if (j < nrow) {
          const float4 st = tv.row_stats[((int64_t)l * dm.G + g) * dm.rows + w * dm.W + j];
          cT[rt][r] = st.x * LOG2E + __log2f(st.y);
        }
      }
  }
  const int64_t c0 = (int64_t)ch * MH_CH;
  int64_t c1 = c0 + MH_CH < dm.N_c ? c0 + MH_CH : dm.N_c;
  if (MODE != RR_DIRECT && (int64_t)umax + 1 < c1) c1 = (int64_t)umax + 1;
  const uint16_t* Kp = K + ((int64_t)l * dm.G + g) * dm.T * D;
  float m[4], z[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) { m[rt] = -INFINITY; z[rt] = 0.f; }
  // the first MH_PF staging rounds of the next sub-chunk are loaded into
  // registers while the current one is computed (all of them for blocks of
  // 256 threads or more at d = 128); further rounds load at store time
  const int bd = blockDim.x;
  uint4 pre[MH_PF];
  auto prefetch = [&](int64_t s0n) {
    const int ntn = (int)(c1 - s0n < MH_SUB ? c1 - s0n : MH_SUB);
#pragma unroll
    for (int q = 0; q < MH_PF; ++q) {
      const int e = tid + bd * q, tt = e / C8, c = e % C8;
      pre[q] = e < MH_SUB * C8 && tt < ntn ? *(const uint4*)(Kp + (s0n + tt) * D + 8 * c) : make_uint4(0, 0, 0, 0);
    }
  };
  if (c0 < c1) prefetch(c0);
  for (int64_t s0 = c0; s0 < c1; s0 += MH_SUB) {
    const int nt = (int)(c1 - s0 < MH_SUB ? c1 - s0 : MH_SUB);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < MH_PF; ++q) {
      const int e = tid + bd * q;
      if (e < MH_SUB * C8) *(uint4*)(sk + (e / C8) * LDK + 8 * (e % C8)) = pre[q];
    }
    for (int e = tid + bd * MH_PF; e < MH_SUB * C8; e += bd) {
      const int tt = e / C8, c = e % C8;
      const uint4 v = tt < nt ? *(const uint4*)(Kp + (s0 + tt) * D + 8 * c) : make_uint4(0, 0, 0, 0);
      *(uint4*)(sk + tt * LDK + 8 * c) = v;
    }
    if (s0 + MH_SUB < c1) prefetch(s0 + MH_SUB);
    __syncthreads();
    for (int tt = 0; tt < MH_SUB / 16; ++tt) {
      if (16 * tt >= nt) break;
      uint4 kf[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) kf[s] = *(const uint4*)(sk + (16 * tt + i16) * LDK + 32 * s + 8 * g4);
      if (MODE == RR_DIRECT) {
        // rows as M, tokens as N: the lane holds rows 16 rt + 4 g4 + r of token
        // s0 + 16 tt + i16, summed in registers and over the four lanes of its
        // column; a token past the chunk (zero key rows) is computed and never
        // read back
        f32x4 acc[4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
          acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < KS; ++s) acc[rt] = mfma_bf16_16x16x32(pk8(qf[rt][s]), pk8(kf[s]), acc[rt]);
        }
        float e[16];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
          for (int r = 0; r < 4; ++r) e[4 * rt + r] = __builtin_amdgcn_exp2f(fmaf(acc[rt][r], sc2, -cT[rt][r]));
#pragma unroll
        for (int w2 = 8; w2 > 0; w2 >>= 1)
#pragma unroll
          for (int i = 0; i < w2; ++i) e[i] += e[i + w2];
        const float sv = col_sum4(e[0]);
        if (g4 == 0) red[w][16 * tt + i16] = sv;
        continue;
      }
      f32x4 acc[4];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) acc[rt] = mfma_bf16_16x16x32(pk8(kf[s]), pk8(qf[rt][s]), acc[rt]);
      }
      // lane holds tokens tb + r of row 16 rt + i16
      const int64_t tb = s0 + 16 * tt + 4 * g4;
      if (MODE == RR_HOP_STATS) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
          float x[4], lm = -INFINITY;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const bool ok = tb + r < c1 && tb + r <= uj[rt];
            x[r] = ok ? acc[rt][r] * sc2 : -INFINITY;
            lm = fmaxf(lm, x[r]);
          }
          if (lm > m[rt]) { z[rt] *= __builtin_amdgcn_exp2f(m[rt] - lm); m[rt] = lm; }
          if (lm != -INFINITY)
#pragma unroll
            for (int r = 0; r < 4; ++r) z[rt] += __builtin_amdgcn_exp2f(x[r] - m[rt]);
        }
      } else {
        float sv[4] = {0.f, 0.f, 0.f, 0.f};
        if (MODE == RR_DIRECT && 16 * tt + 16 <= nt) {
          // direct pass, no token past the chunk: every row sees every token
          // (weight 1) and the masked rows add 0
#pragma unroll
          for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int r = 0; r < 4; ++r) sv[r] += __builtin_amdgcn_exp2f(fmaf(acc[rt][r], sc2, -cj[rt]));
        } else {
#pragma unroll
          for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool ok = tb + r < c1 && tb + r <= uj[rt];
              const float v = wj[rt] * __builtin_amdgcn_exp2f(acc[rt][r] * sc2 - cj[rt]);
              sv[r] += ok ? v : 0.f;
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) sv[r] = row_sum16(sv[r]);
        if (i16 < 4) red[w][16 * tt + 4 * g4 + i16] = i16 == 0 ? sv[0] : i16 == 1 ? sv[1] : i16 == 2 ? sv[2] : sv[3];
      }
    }
    if (MODE != RR_HOP_STATS) {
      __syncthreads();
      if (tid < nt) {
        float s = 0.f;
        for (int w2 = 0; w2 < nw; ++w2) s += red[w2][tid];
        if (MODE == RR_HOP_SUMS) {
          mh.dpart[(int64_t)grp * dm.N_c + s0 + tid] = s;
        } else {
          const int lg = l * dm.G + g;
          tv.tok_R[(int64_t)lg * dm.N_c + s0 + tid] = s / (tv.lg_S[lg] + dm.eps);
        }
      }
    }
  }
  if (MODE == RR_HOP_STATS) {
    // merge the four lanes of each row (lanes i16 + 16 k)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
#pragma unroll
      for (int o = 16; o < 64; o <<= 1) {
        const float m2 = __shfl_xor(m[rt], o, 64), z2 = __shfl_xor(z[rt], o, 64);
        const float mn = fmaxf(m[rt], m2);
        if (mn != -INFINITY) {
          z[rt] = z[rt] * __builtin_amdgcn_exp2f(m[rt] - mn) + z2 * __builtin_amdgcn_exp2f(m2 - mn);
          m[rt] = mn;
        }
      }
      if (g4 == 0) {
        const int ngrp = dm.n_gl * dm.G;
        mh.rpart[((int64_t)ch * ngrp + grp) * rmax + w * MH_SEEDS + 16 * rt + i16] = make_float2(m[rt], z[rt]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp32: one thread per row r = 64 hl + j on the vector ALUs (hop passes only).
// ---------------------------------------------------------------------------
template <int D, int PASS>
__global__ __launch_bounds__(256) void k_mh_rows(Dims dm, const float* __restrict__ K, const float* __restrict__ Qg,
                                                 MhView mh) {
  __shared__ __align__(16) float sk[MH_SUB * D];
  __shared__ float red[4][MH_SUB];
  const int ch = blockIdx.x, grp = blockIdx.y, zb = blockIdx.z;
  const int gi = grp / dm.G, g = grp % dm.G;
  const int l = dm.gl[gi];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rmax = dm.hpg * MH_SEEDS;
  const int nz = (rmax + 255) / 256;
  const int r = zb * 256 + tid;
  const int hl = r / MH_SEEDS, j = r % MH_SEEDS;
  const int ns = *mh.ns;
  const bool on = hl < dm.hpg && j < ns;
  float q[D];
  int u = -1;
  float w = 0.f;
  if (on) {
    u = mh.seeds[j];
    w = mh.wts[j];
    const float* qr = Qg + (((int64_t)gi * dm.H + g * dm.hpg + hl) * dm.T + u) * D;
    const float sc2 = LOG2E / sqrtf((float)D);
#pragma unroll
    for (int k = 0; k < D; ++k) q[k] = qr[k] * sc2;
  } else {
#pragma unroll
    for (int k = 0; k < D; ++k) q[k] = 0.f;
  }
  int umax = -1;
  for (int s = 0; s < ns; ++s) umax = max(umax, mh.seeds[s]);
  const int64_t c0 = (int64_t)ch * MH_CH;
  const int64_t c1 = min((int64_t)umax + 1, min(c0 + MH_CH, dm.N_c));
  const float* Kp = K + ((int64_t)l * dm.G + g) * dm.T * D;
  float2 st = make_float2(0.f, 0.f);
  if (PASS == 1 && on) st = mh.rstat[(int64_t)grp * rmax + r];
  float m = -INFINITY, zs = 0.f;
  for (int64_t s0 = c0; s0 < c1; s0 += MH_SUB) {
    const int nt = (int)min((int64_t)MH_SUB, c1 - s0);
    __syncthreads();
    for (int e = tid; e < MH_SUB * D; e += 256) {
      const int tt = e / D, k = e % D;
      sk[e] = tt < nt ? Kp[(s0 + tt) * D + k] : 0.f;
    }
    __syncthreads();
    for (int tt = 0; tt < nt; ++tt) {
      const int64_t t = s0 + tt;
      float x = 0.f;
#pragma unroll
      for (int k = 0; k < D; k += 4) {
        const float4 kv = *(const float4*)(sk + tt * D + k);
        x += q[k] * kv.x + q[k + 1] * kv.y + q[k + 2] * kv.z + q[k + 3] * kv.w;
      }
      const bool vis = on && t <= u;
      if (PASS == 0) {
        if (vis) {
          const float mn = fmaxf(m, x);
          zs = zs * __builtin_amdgcn_exp2f(m - mn) + __builtin_amdgcn_exp2f(x - mn);
          m = mn;
        }
      } else {
        float v = vis ? w * __builtin_amdgcn_exp2f(x - st.x - st.y) : 0.f;
        v = wave_sum_dpp(v);
        if (lane == 0) red[wave][tt] = v;
      }
    }
    if (PASS == 1) {
      __syncthreads();
      if (tid < nt)
        mh.dpart[((int64_t)grp * nz + zb) * dm.N_c + s0 + tid] =
            (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
    }
  }
  if (PASS == 0 && r < rmax) {
    const int ngrp = dm.n_gl * dm.G;
    mh.rpart[((int64_t)ch * ngrp + grp) * rmax + r] = make_float2(m, zs);
  }
}

// merges the chunk partials of every row: (max, log2 of the partition sum)
__global__ void k_mh_rowstat_combine(Dims dm, MhView mh, int nch) {
  const int rmax = dm.hpg * MH_SEEDS;
  const int ngrp = dm.n_gl * dm.G;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)ngrp * rmax) return;
  float m = -INFINITY, z = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float2 p = mh.rpart[(int64_t)c * ngrp * rmax + i];
    if (p.x == -INFINITY) continue;
    const float mn = fmaxf(m, p.x);
    z = z * __builtin_amdgcn_exp2f(m - mn) + p.y * __builtin_amdgcn_exp2f(p.x - mn);
    m = mn;
  }
  mh.rstat[i] = make_float2(m, z > 0.f ? __log2f(z) : 0.f);
}

// d^(k) over layers, heads and row blocks; zero at every seed so far; accumulated
__global__ void k_mh_hop_reduce(Dims dm, MhView mh, int hop, int nz) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= dm.N_c) return;
  const int ngrp = dm.n_gl * dm.G;
  const int ns = *mh.ns;
  int umax = -1;                              // tokens past the furthest seed have no partials
  for (int s = 0; s < ns; ++s) umax = max(umax, mh.seeds[s]);
  float d = 0.f;
  if (t <= umax)
    for (int k = 0; k < ngrp * nz; ++k) d += mh.dpart[(int64_t)k * dm.N_c + t];
  const int nu = *mh.nused;
  for (int k = 0; k < nu; ++k)
    if (mh.used[k] == t) d = 0.f;
  mh.dk[t] = d;
  float decay = 1.f;
  for (int k = 0; k < hop; ++k) decay *= MH_RHO;
  mh.dacc[t] = (hop == 0 ? 0.f : mh.dacc[t]) + decay * d;
}

__global__ __launch_bounds__(1024) void k_mh_finish(Dims dm, MhView mh) {
  __shared__ double sred[16];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  double a = 0.0;
  for (int64_t t = tid; t < dm.N_c; t += 1024) a += mh.dacc[t];
  a = wave_sum(a);
  if (lane == 0) sred[wave] = a;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < 16; ++w) s += sred[w];
  const float inv = (float)(1.0 / (s + (double)dm.eps));
  for (int64_t t = tid; t < dm.N_c; t += 1024) mh.dhat[t] = mh.dacc[t] * inv;
}

static void mh_seeds(const Dims& dm, const MhView& mh, hipStream_t st) {
  const unsigned nb = (unsigned)((dm.N_c + MH_TOPB - 1) / MH_TOPB);
  hipLaunchKernelGGL(k_mh_top, dim3(nb), dim3(256), 0, st, dm, mh);
  hipLaunchKernelGGL(k_mh_seeds, dim3(1), dim3(1024), 0, st, dm, mh);
}

template <int D>
static hipError_t mh_bf16(const Dims& dm, const uint16_t* K, const uint16_t* Q, const uint16_t* Qg,
                          const TreeView& tv, const MhView& mh, hipStream_t st) {
  const int rmax = dm.hpg * MH_SEEDS;
  const int ngrp = dm.n_gl * dm.G;
  const unsigned nch = (unsigned)((dm.N_c + MH_CH - 1) / MH_CH);
  const unsigned tb = (unsigned)((dm.N_c + 255) / 256);
  const dim3 blk(64 * dm.hpg);
  (void)Q;                                    // s-hat is in the token values (launch_token_relevance)
  hipLaunchKernelGGL(k_mh_seed_score, dim3(tb), dim3(256), 0, st, dm, tv, mh);
  for (int hop = 0; hop < MH_HOPS; ++hop) {
    mh_seeds(dm, mh, st);
    hipLaunchKernelGGL((k_rel_rows<D, RR_HOP_STATS>), dim3(nch, ngrp), blk, 0, st, dm, K, Qg, tv, mh);
    hipLaunchKernelGGL(k_mh_rowstat_combine, dim3((unsigned)((ngrp * rmax + 255) / 256)), dim3(256), 0, st, dm, mh,
                       (int)nch);
    hipLaunchKernelGGL((k_rel_rows<D, RR_HOP_SUMS>), dim3(nch, ngrp), blk, 0, st, dm, K, Qg, tv, mh);
    hipLaunchKernelGGL(k_mh_hop_reduce, dim3(tb), dim3(256), 0, st, dm, mh, hop, 1);
  }
  hipLaunchKernelGGL(k_mh_finish, dim3(1), dim3(1024), 0, st, dm, mh);
  return hipGetLastError();
}

template <int D>
static hipError_t mh_f32(const Dims& dm, const float* K, const float* Qg, const TreeView& tv, const MhView& mh,
                         hipStream_t st) {
  const int rmax = dm.hpg * MH_SEEDS;
  const int ngrp = dm.n_gl * dm.G;
  const int nz = (rmax + 255) / 256;
  const unsigned nch = (unsigned)((dm.N_c + MH_CH - 1) / MH_CH);
  const unsigned tb = (unsigned)((dm.N_c + 255) / 256);
  hipLaunchKernelGGL(k_mh_seed_score, dim3(tb), dim3(256), 0, st, dm, tv, mh);
  for (int hop = 0; hop < MH_HOPS; ++hop) {
    mh_seeds(dm, mh, st);
    hipLaunchKernelGGL((k_mh_rows<D, 0>), dim3(nch, ngrp, nz), dim3(256), 0, st, dm, K, Qg, mh);
    hipLaunchKernelGGL(k_mh_rowstat_combine, dim3((unsigned)((ngrp * rmax + 255) / 256)), dim3(256), 0, st, dm, mh,
                       (int)nch);
    hipLaunchKernelGGL((k_mh_rows<D, 1>), dim3(nch, ngrp, nz), dim3(256), 0, st, dm, K, Qg, mh);
    hipLaunchKernelGGL(k_mh_hop_reduce, dim3(tb), dim3(256), 0, st, dm, mh, hop, nz);
  }
  hipLaunchKernelGGL(k_mh_finish, dim3(1), dim3(1024), 0, st, dm, mh);
  return hipGetLastError();
}

// The direct relevance s-hat of every (l, g, t) into the token values (bf16
// caches, hpg <= 8): the pass-2 sums of eq:app_direct_relevance over the hpg W
// window-query rows, each normalised by its row statistics, divided by S_{l,g}.
hipError_t launch_token_relevance(const Dims& dm, const void* K, const void* Q, const TreeView& tv, hipStream_t st) {
  if (!token_relevance_pass(dm)) return hipErrorInvalidValue;
  if (dm.N_c <= 0) return hipSuccess;
  const MhView none{};
  const dim3 grid((unsigned)((dm.N_c + MH_CH - 1) / MH_CH), (unsigned)(dm.L * dm.G)), blk(64 * dm.hpg);
  if (dm.d == 128)
    hipLaunchKernelGGL((k_rel_rows<128, RR_DIRECT>), grid, blk, 0, st, dm, (const uint16_t*)K, (const uint16_t*)Q, tv, none);
  else if (dm.d == 64)
    hipLaunchKernelGGL((k_rel_rows<64, RR_DIRECT>), grid, blk, 0, st, dm, (const uint16_t*)K, (const uint16_t*)Q, tv, none);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_multihop(const Dims& dm, const void* K, const void* Q, const void* Q_graph, const TreeView& tv,
                           void* mh_base, hipStream_t st) {
  const MhView mh = mh_view(mh_base, dm);
  if (dm.N_c <= 0) return hipSuccess;
  if (dm.hpg < 1 || dm.hpg > 8 || dm.W > MH_SEEDS) return hipErrorInvalidValue;
  if (dm.dtype == GRACEKV_BF16) {
    const uint16_t *k = (const uint16_t*)K, *q = (const uint16_t*)Q, *qg = (const uint16_t*)Q_graph;
    if (dm.d == 128) return mh_bf16<128>(dm, k, q, qg, tv, mh, st);
    if (dm.d == 64) return mh_bf16<64>(dm, k, q, qg, tv, mh, st);
  } else if (dm.d == 64) {
    return mh_f32<64>(dm, (const float*)K, (const float*)Q_graph, tv, mh, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace gkv
