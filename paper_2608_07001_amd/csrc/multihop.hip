// Multi-hop relevance (App. A.4 eq:app_global_seed_score,
// eq:app_hop_propagation, eq:app_diffused_relevance, eq:app_bottom_up_value).
//
// Runs inside gracekv_build_trees when lambda_graph > 0, after a first pass of
// the root kernel has written the direct relevance s-hat of every (l, g) into
// the token-value array:
//   * k_mh_seed_score: S_t = mean over (l, g) of s-hat_{l,g,t};
//   * k_mh_seeds (one workgroup): positions in descending score (ties to the
//     smaller position) while their cumulative share of the total stays below
//     0.9 (the one reaching it included), at most 64, weights proportional to
//     the score;
//   * k_mh_rows, pass 0 and 1, grid (token chunk, propagation layer x KV head,
//     row block): one thread per row (query head of the group x seed) holds
//     the seed's query of that layer and head in registers; 64-token blocks of
//     keys are staged in LDS.  Pass 0 gives each row's maximum and partition
//     sum over its causal range [0, u]; pass 1 sums w_u pi_{u,t} over the rows
//     for every token of C;
//   * k_mh_hop_reduce: d^(k)_t over layers and heads, zero at the current and
//     earlier seeds, accumulated with the decay 0.5^(k-1);
//   * k_mh_finish: d-hat = d / (sum_C d + eps).
// The root kernel then runs again and mixes R^tok = (1 - lambda) s-hat +
// lambda d-hat.
#include "common.h"

namespace gkv {

constexpr int MH_SEEDS = 64;                 // at most this many seeds per hop
constexpr int MH_HOPS = 2;
constexpr int MH_CH = 1024;                  // tokens per workgroup of the row passes
constexpr int MH_SUB = 64;                   // tokens staged at once
constexpr double MH_ETA = 0.9;               // cumulative seed share
constexpr float MH_RHO = 0.5f;               // inter-hop decay

static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

MhView mh_view(void* base, const Dims& dm) {
  char* p = (char*)base;
  MhView v;
  const size_t N = (size_t)dm.N_c;
  const int rmax = dm.hpg * MH_SEEDS;
  const int ngrp = dm.n_gl * dm.G;
  const int nz = (rmax + 255) / 256;
  const int nch = (int)((N + MH_CH - 1) / MH_CH);
  v.dk = (float*)p; p += al(N * 4);
  v.dacc = (float*)p; p += al(N * 4);
  v.dhat = (float*)p; p += al(N * 4);
  v.seeds = (int32_t*)p; p += al(MH_SEEDS * 4);
  v.wts = (float*)p; p += al(MH_SEEDS * 4);
  v.ns = (int32_t*)p; p += al(16);
  v.used = (int32_t*)p; p += al(MH_HOPS * MH_SEEDS * 4);
  v.nused = (int32_t*)p; p += al(16);
  v.rstat = (float2*)p; p += al((size_t)ngrp * rmax * 8);
  v.rpart = (float2*)p; p += al((size_t)nch * ngrp * rmax * 8);
  v.dpart = (float*)p; p += al((size_t)ngrp * nz * N * 4);
  v.bytes = (size_t)(p - (char*)base);
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

__global__ __launch_bounds__(1024) void k_mh_seeds(Dims dm, MhView mh) {
  __shared__ double sred[16];
  __shared__ unsigned long long skey[16];
  __shared__ double tot;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const float* sc = mh.dk;
  double a = 0.0;
  for (int64_t t = tid; t < dm.N_c; t += 1024) a += sc[t];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) a += __shfl_xor(a, o, 64);
  if (lane == 0) sred[wave] = a;
  __syncthreads();
  if (tid == 0) {
    double s = 0.0;
    for (int w = 0; w < 16; ++w) s += sred[w];
    tot = s;
  }
  __syncthreads();
  const double total = tot;
  uint64_t prev = ~0ull;
  double cum = 0.0, wsum = 0.0;
  int ns = 0;
  for (int k = 0; k < MH_SEEDS; ++k) {
    if (!(total > 0.0) || cum >= MH_ETA) break;
    uint64_t best = 0;
    for (int64_t t = tid; t < dm.N_c; t += 1024) {
      const uint64_t key = mh_key(sc[t], t);
      if (key < prev && key > best) best = key;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint64_t b2 = __shfl_xor(best, o, 64);
      best = b2 > best ? b2 : best;
    }
    if (lane == 0) skey[wave] = best;
    __syncthreads();
    uint64_t b = skey[0];
    for (int w = 1; w < 16; ++w) b = skey[w] > b ? skey[w] : b;
    __syncthreads();
    const float s = __uint_as_float((uint32_t)(b >> 32));
    if (!(s > 0.f)) break;
    const int t = (int)(0xFFFFFFFFu - (uint32_t)(b & 0xFFFFFFFFu));
    if (tid == 0) { mh.seeds[ns] = t; mh.wts[ns] = s; }
    cum += (double)s / total;
    wsum += (double)s;
    ++ns;
    prev = b;
  }
  __syncthreads();
  if (tid < ns) {
    mh.wts[tid] = (float)((double)mh.wts[tid] / wsum);
    mh.used[*mh.nused + tid] = mh.seeds[tid];
  }
  __syncthreads();
  if (tid == 0) { *mh.ns = ns; *mh.nused += ns; }
}

// the seed query of row r (head slot r / ns, seed r % ns), scaled to base-2 logits
template <typename T, int D>
__device__ __forceinline__ bool mh_row(const Dims& dm, const T* __restrict__ Qg, const MhView& mh, int gi, int g,
                                       int r, float* q, int& u, float& w) {
  const int ns = *mh.ns;
  if (ns == 0 || r >= dm.hpg * ns) return false;
  const int hl = r / ns, s = r % ns;
  u = mh.seeds[s];
  w = mh.wts[s];
  const int h = g * dm.hpg + hl;
  const T* qr = Qg + (((int64_t)gi * dm.H + h) * dm.T + u) * D;
  const float sc2 = 1.44269504088896341f / sqrtf((float)D);
#pragma unroll
  for (int k = 0; k < D; ++k) q[k] = ldf(qr, k) * sc2;
  return true;
}

template <typename T, int D, int PASS>
__global__ __launch_bounds__(256) void k_mh_rows(Dims dm, const T* __restrict__ K, const T* __restrict__ Qg,
                                                 MhView mh) {
  __shared__ __align__(16) float sk[MH_SUB * D];
  __shared__ float red[4][MH_SUB];
  const int ch = blockIdx.x, grp = blockIdx.y, z = blockIdx.z;
  const int gi = grp / dm.G, g = grp % dm.G;
  const int l = dm.gl[gi];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rmax = dm.hpg * MH_SEEDS;
  const int r = z * 256 + tid;
  float q[D];
  int u = -1;
  float w = 0.f;
  const bool on = mh_row<T, D>(dm, Qg, mh, gi, g, r, q, u, w);
  // the furthest seed bounds the tokens any row sees
  int umax = -1;
  for (int s = 0; s < *mh.ns; ++s) umax = max(umax, mh.seeds[s]);
  const int64_t c0 = (int64_t)ch * MH_CH;
  const int64_t c1 = min((int64_t)umax + 1, min(c0 + MH_CH, dm.N_c));
  const T* Kp = K + ((int64_t)l * dm.G + g) * dm.T * D;
  float2 st = make_float2(0.f, 0.f);
  if (PASS == 1 && on) st = mh.rstat[(int64_t)grp * rmax + r];
  float m = -INFINITY, zs = 0.f;
  for (int64_t s0 = c0; s0 < c1; s0 += MH_SUB) {
    const int nt = (int)min((int64_t)MH_SUB, c1 - s0);
    __syncthreads();
    for (int e = tid; e < MH_SUB * D; e += 256) {
      const int tt = e / D, k = e % D;
      sk[e] = tt < nt ? ldf(Kp + (s0 + tt) * D, k) : 0.f;
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
      if (tid < nt) {
        const int nz = (rmax + 255) / 256;
        mh.dpart[((int64_t)grp * nz + z) * dm.N_c + s0 + tid] =
            (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
      }
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
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) a += __shfl_xor(a, o, 64);
  if (lane == 0) sred[wave] = a;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < 16; ++w) s += sred[w];
  const float inv = (float)(1.0 / (s + (double)dm.eps));
  for (int64_t t = tid; t < dm.N_c; t += 1024) mh.dhat[t] = mh.dacc[t] * inv;
}

template <typename T, int D>
static hipError_t mh_hops(const Dims& dm, const T* K, const T* Qg, const TreeView& tv, const MhView& mh,
                          hipStream_t st) {
  const int rmax = dm.hpg * MH_SEEDS;
  const int ngrp = dm.n_gl * dm.G;
  const int nz = (rmax + 255) / 256;
  const int nch = (int)((dm.N_c + MH_CH - 1) / MH_CH);
  const unsigned tb = (unsigned)((dm.N_c + 255) / 256);
  hipLaunchKernelGGL(k_mh_seed_score, dim3(tb), dim3(256), 0, st, dm, tv, mh);
  for (int hop = 0; hop < MH_HOPS; ++hop) {
    hipLaunchKernelGGL(k_mh_seeds, dim3(1), dim3(1024), 0, st, dm, mh);
    hipLaunchKernelGGL((k_mh_rows<T, D, 0>), dim3(nch, ngrp, nz), dim3(256), 0, st, dm, K, Qg, mh);
    hipLaunchKernelGGL(k_mh_rowstat_combine, dim3((unsigned)((ngrp * rmax + 255) / 256)), dim3(256), 0, st, dm, mh,
                       nch);
    hipLaunchKernelGGL((k_mh_rows<T, D, 1>), dim3(nch, ngrp, nz), dim3(256), 0, st, dm, K, Qg, mh);
    hipLaunchKernelGGL(k_mh_hop_reduce, dim3(tb), dim3(256), 0, st, dm, mh, hop, nz);
  }
  hipLaunchKernelGGL(k_mh_finish, dim3(1), dim3(1024), 0, st, dm, mh);
  return hipGetLastError();
}

hipError_t launch_multihop(const Dims& dm, const void* K, const void* Q_graph, const TreeView& tv, void* mh_base,
                           hipStream_t st) {
  const MhView mh = mh_view(mh_base, dm);
  if (dm.N_c <= 0) return hipSuccess;
  if (dm.dtype == GRACEKV_BF16) {
    if (dm.d == 128) return mh_hops<uint16_t, 128>(dm, (const uint16_t*)K, (const uint16_t*)Q_graph, tv, mh, st);
    if (dm.d == 64) return mh_hops<uint16_t, 64>(dm, (const uint16_t*)K, (const uint16_t*)Q_graph, tv, mh, st);
  } else if (dm.d == 64) {
    return mh_hops<float, 64>(dm, (const float*)K, (const float*)Q_graph, tv, mh, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace gkv
