// Refinement below the roots, one depth at a time (bf16 caches; App. A.3
// "Recursive refinement rule", App. B.4 eq:app_tree_split_candidates).
//
// The nodes of a unit are numbered in BFS order: the root, then its children,
// then the children of node 1 in order, and so on.  That is depth order, and
// within a depth the order of the parents.  So every node of one depth can be
// refined at the same time, by the root-split kernel in its level mode, which
// writes one result per node (kind, cut, children with D and R, the Split's
// utility), and a level pass then numbers the children: one wave per unit walks
// the unit's nodes of that depth (at most NMAX of them, two per lane) in order,
// gives each refined node its first child index by a prefix sum over the child
// counts, writes parents, children and (pruned build) the Split keys, and lists
// the children to refine at the next depth as one contiguous block of items per
// unit, in BFS order.  A node is refined when it has two or more tokens and
// (pruned build) the effective key of the op that creates it reaches theta,
// the rule of the per-unit refinement kernel, which takes over below the last
// depth done here and continues from the same node table.
//
// Counters (lv_ctr): [d & 1] items of depth d; [2] next item of the split
// kernel; [4 + (d & 1)] units with items at depth d; [8] the unit capacity.
// The split kernel of depth d clears the counters of depth d + 1; the level
// pass of depth d clears the split kernel's cursor.
#include <cstdlib>

#include "common.h"

namespace gkv {

int64_t level_capacity(int64_t LG, int64_t N_c) { return LG * (N_c / 2) + 1; }

static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t level_region_bytes(int64_t LG, int64_t N_c, int64_t unit_cap) {
  const size_t cap = (size_t)level_capacity(LG, N_c);
  return al256(cap * 32) + al256(cap * 48) + al256((size_t)unit_cap * 8) + al256((size_t)unit_cap * 16) + al256(64);
}

__global__ void k_level_reset(const TreeView* __restrict__ tvp, int ucap) {
  const TreeView& tv = *tvp;
  if (threadIdx.x < 16) tv.lv_ctr[threadIdx.x] = threadIdx.x == 8 ? ucap : 0;
}

// exclusive prefix over the wave (lane order) and the wave total
__device__ __forceinline__ int wave_excl(int v, int& total) {
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if ((int)(threadIdx.x & 63) >= o) x += y;
  }
  total = __shfl(x, 63, 64);
  return x - v;
}

// The units with nodes at depth lvl (>= 1): children numbered and placed, depth
// lvl + 1 listed.
__global__ __launch_bounds__(256) void k_level(const Dims* __restrict__ dmp, const TreeView* __restrict__ tvp, int lvl,
                                               int full) {
  const Dims& dm = *dmp;
  const TreeView& tv = *tvp;
  const int lane = threadIdx.x & 63;
  const int P = lvl & 1, Pn = (lvl + 1) & 1;
  if (blockIdx.x == 0 && threadIdx.x == 0) tv.lv_ctr[2] = 0;   // the next split kernel's cursor
  const int nunits = __builtin_amdgcn_readfirstlane(tv.lv_ctr[4 + P]);
  const int J = *tv.nslots;
  const uint64_t theta = full ? 0ull : tv.theta[0];
  const int64_t ucap = (int64_t)dm.L * dm.G * dm.J_cap;
  // wave w takes units w, w + W, ... (W waves in the grid): the loop head has
  // no lane-dependent branch.  (A cursor taken by lane 0 and broadcast by a
  // lane shuffle at the head would let the compiler send lanes 1-63 round the
  // loop again before lane 0 had taken the next index: they would read its old
  // one for ever.)
  const int nw = (int)gridDim.x * (int)(blockDim.x >> 6);
  for (int k = __builtin_amdgcn_readfirstlane((int)blockIdx.x * (int)(blockDim.x >> 6) + (int)(threadIdx.x >> 6));
       k < nunits; k += nw) {
    do {
    const int64_t unit = tv.lv_units[(int64_t)P * ucap + k];
    const int lg = (int)(unit / dm.J_cap), j = (int)(unit % dm.J_cap);
    if (j >= J) break;
    const int a0 = tv.slots[j];
    const int nslot = tv.slots[j + 1] - a0;
    const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)a0;
    const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
    const int32_t w_bits = __float_as_int(tv.omega[lg]);
    const int cnt = tv.unit_nn[unit];
    // this depth's nodes [lo, hi) with their items from ib
    const int4 st = tv.lv_state[unit];
    const int lo = st.x, hi = st.y, ib = st.z;
    // per lane: two nodes i = lo + lane + 64 h; refined ones read their result
    int nk[2] = {0, 0}, nx[2] = {0, 0};
    int4 r0[2], r1[2], r2[2];
    uint64_t Ech[2] = {0ull, 0ull};
    int ai[2] = {0, 0};
    int rank_base = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      r0[h] = r1[h] = r2[h] = make_int4(0, 0, 0, 0);
      const int i = lo + lane + 64 * h;
      bool ref = false;
      uint64_t Ei = 0ull;
      if (i < hi) {
        const int64_t s = base + i;
        ai[h] = tv.node_a[s];
        if (tv.node_nch[s] == 0 && tv.node_n[s] >= 2) {
          if (!full) {
            const int par = tv.node_parent[s];
            Ei = par < 0 ? tv.add_E[unit] : tv.sp_E[base + par];
          }
          ref = full || Ei >= theta;
        }
      }
      const uint64_t m = __ballot(ref);
      const int rank = rank_base + __popcll(m & ((1ull << lane) - 1ull));
      rank_base += __popcll(m);
      if (ref && (int64_t)ib + rank < tv.lv_cap) {
        const int4* r = (const int4*)(tv.lv_res + 12 * (int64_t)(ib + rank));
        r0[h] = r[0]; r1[h] = r[1]; r2[h] = r[2];
        nk[h] = (r0[h].x >> 8) & 255;
        if (nk[h] < 2 || nk[h] > 3) nk[h] = 0;   // not a result of this depth's split pass
        if (!full) {
          const uint64_t kk = op_key(__int_as_float(r0[h].y), ord * 256u + 1u + (uint32_t)i);
          Ech[h] = kk < Ei ? kk : Ei;
        }
        const int kn0 = r0[h].z >> 16, kn1 = r0[h].w >> 16, kn2 = r1[h].x >> 16;
        const bool pass = full || Ech[h] >= theta;
        nx[h] = pass ? (int)(kn0 >= 2) + (int)(kn1 >= 2) + (int)(nk[h] > 2 && kn2 >= 2) : 0;
      }
    }
    int tk0, tk1, tx0, tx1;
    const int ck0 = wave_excl(nk[0], tk0), ck1 = wave_excl(nk[1], tk1);
    const int cx0 = wave_excl(nx[0], tx0), cx1 = wave_excl(nx[1], tx1);
    const int newcnt = cnt + tk0 + tk1;
    const int ktot = tx0 + tx1;
    int nbl = 0;
    if (lane == 0 && ktot > 0) nbl = atomicAdd(&tv.lv_ctr[Pn], ktot);
    const int nb = __builtin_amdgcn_readfirstlane(__shfl(nbl, 0, 64));
    // neither can happen (the nodes of a depth are disjoint, a tree over n tokens
    // has at most 2n - 1 nodes); checked so that no write leaves the unit's range
    if ((ktot > 0 && (int64_t)nb + ktot > tv.lv_cap) || newcnt > 2 * nslot - 1) {
      if (lane == 0) atomicOr(tv.status, STATUS_CAPACITY);
      break;
    }
    auto put_item = [&](int pos, int c, int a_abs, int n, float Dc, float Rc, uint64_t E) {
      int4* it = (int4*)(tv.lv_items + 8 * (int64_t)pos);
      it[0] = make_int4((int32_t)unit, a_abs, n | (c << 16), __float_as_int(Dc));
      it[1] = make_int4(__float_as_int(Rc), w_bits, (int32_t)(uint32_t)E, (int32_t)(uint32_t)(E >> 32));
    };
    {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (nk[h] == 0) continue;
        const int i = lo + lane + 64 * h;
        const int64_t s = base + i;
        const int fc = cnt + (h == 0 ? ck0 : tk0 + ck1);
        int xi = nb + (h == 0 ? cx0 : tx0 + cx1);
        const int kind = r0[h].x & 255, cut = r0[h].x >> 16;
        tv.node_child[s] = fc;
        tv.node_nch[s] = (uint8_t)nk[h];
        tv.node_kind[s] = (uint8_t)kind;
        tv.node_cut[s] = ai[h] + cut;
        if (!full) {
          tv.sp_U[s] = __int_as_float(r0[h].y);
          tv.sp_E[s] = Ech[h];
          tv.sp_cost[s] = (uint8_t)(nk[h] - 1);
          tv.sp_exec[s] = 0;
        }
        const int kw[3] = {r0[h].z, r0[h].w, r1[h].x};
        const int kD[3] = {r1[h].y, r1[h].z, r1[h].w};
        const int kR[3] = {r2[h].x, r2[h].y, r2[h].z};
        const bool pass = full || Ech[h] >= theta;
        for (int c = 0; c < nk[h]; ++c) {
          const int64_t sc = base + fc + c;
          const int ka = kw[c] & 0xffff, kn = kw[c] >> 16;
          tv.node_a[sc] = ai[h] + ka;
          tv.node_n[sc] = kn;
          tv.node_child[sc] = -1;
          tv.node_parent[sc] = i;
          tv.node_nch[sc] = 0;
          tv.node_kind[sc] = 0;
          tv.node_cut[sc] = -1;
          tv.node_D[sc] = __int_as_float(kD[c]);
          tv.node_R[sc] = __int_as_float(kR[c]);
          tv.sp_cost[sc] = 0;
          tv.sp_exec[sc] = 0;
          if (!full) { tv.sp_U[sc] = 0.f; tv.sp_E[sc] = 0ull; }
          if (pass && kn >= 2) {
            put_item(xi, fc + c, ai[h] + ka, kn, __int_as_float(kD[c]), __int_as_float(kR[c]), Ech[h]);
            ++xi;
          }
        }
      }
    }
    if (lane == 0) {
      tv.unit_nn[unit] = newcnt;
      tv.lv_state[unit] = make_int4(cnt, newcnt, nb, ktot);
      if (ktot > 0) {
        const int pos = atomicAdd(&tv.lv_ctr[4 + Pn], 1);
        tv.lv_units[(int64_t)Pn * ucap + pos] = (int32_t)unit;
      }
    }
    } while (0);
  }
}

// Depth 1: the children of every root the root pass refined, one unit per
// lane; the wave takes one block of items and one block of list entries.
__global__ __launch_bounds__(256) void k_level_first(const Dims* __restrict__ dmp, const TreeView* __restrict__ tvp,
                                                     int full) {
  const Dims& dm = *dmp;
  const TreeView& tv = *tvp;
  const int lane = threadIdx.x & 63;
  if (blockIdx.x == 0 && threadIdx.x == 0) tv.lv_ctr[2] = 0;   // the next split kernel's cursor
  const int nunits = __builtin_amdgcn_readfirstlane(tv.wctr[0]);
  const int J = *tv.nslots;
  const uint64_t theta = full ? 0ull : tv.theta[0];
  const int64_t ucap = (int64_t)dm.L * dm.G * dm.J_cap;
  const int stride = (int)gridDim.x * (int)blockDim.x;
  for (int k0 = __builtin_amdgcn_readfirstlane((int)blockIdx.x * (int)blockDim.x + (int)(threadIdx.x & ~63u));
       k0 < nunits; k0 += stride) {
    const int k = k0 + lane;
    int64_t unit = 0, base = 0;
    int cnt = 0, m = 0;
    uint64_t Ef = 0ull;
    bool ok[3] = {false, false, false};
    if (k < nunits) {
      unit = tv.work[8 * (int64_t)k];
      const int lg = (int)(unit / dm.J_cap), j = (int)(unit % dm.J_cap);
      if (j < J) {
        base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)tv.slots[j];
        cnt = tv.unit_nn[unit];
        if (!full && cnt > 1) Ef = tv.sp_E[base];   // the root's Split (written by the root pass)
#pragma unroll
        for (int c = 0; c < 3; ++c) {
          ok[c] = 1 + c < cnt && tv.node_n[base + 1 + c] >= 2 && (full || Ef >= theta);
          m += ok[c] ? 1 : 0;
        }
      }
    }
    int tot;
    const int ex = wave_excl(m, tot);
    int nbl = 0;
    if (lane == 0 && tot > 0) nbl = atomicAdd(&tv.lv_ctr[1], tot);
    const int nb = __builtin_amdgcn_readfirstlane(__shfl(nbl, 0, 64));
    const uint64_t has = __ballot(m > 0);
    int ubl = 0;
    if (lane == 0 && has) ubl = atomicAdd(&tv.lv_ctr[5], __popcll(has));
    const int ub = __builtin_amdgcn_readfirstlane(__shfl(ubl, 0, 64));
    const bool fits = (int64_t)nb + tot <= tv.lv_cap;   // always (the roots' children are disjoint)
    if (!fits && lane == 0) atomicOr(tv.status, STATUS_CAPACITY);
    if (fits && m > 0) {
      int xi = nb + ex;
      const int32_t w_bits = __float_as_int(tv.omega[unit / dm.J_cap]);
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        if (!ok[c]) continue;
        const int64_t s = base + 1 + c;
        int4* it = (int4*)(tv.lv_items + 8 * (int64_t)xi);
        it[0] = make_int4((int32_t)unit, tv.node_a[s], tv.node_n[s] | ((1 + c) << 16), __float_as_int(tv.node_D[s]));
        it[1] = make_int4(__float_as_int(tv.node_R[s]), w_bits, (int32_t)(uint32_t)Ef, (int32_t)(uint32_t)(Ef >> 32));
        ++xi;
      }
      tv.lv_state[unit] = make_int4(1, cnt, nb + ex, m);
      tv.lv_units[ucap + ub + __popcll(has & ((1ull << lane) - 1ull))] = (int32_t)unit;
    }
  }
}

// Below the last depth done here: the units still holding nodes to refine
// become the per-unit kernel's work list.
__global__ void k_level_handoff(const TreeView* __restrict__ tvp, int levels) {
  const TreeView& tv = *tvp;
  const int64_t ucap = (int64_t)tv.lv_ctr[8];
  const int P = (levels + 1) & 1;
  const int n = tv.lv_ctr[4 + P];
  for (int i = threadIdx.x; i < n; i += blockDim.x) tv.work[8 * (int64_t)i] = tv.lv_units[P * ucap + i];
  if (threadIdx.x == 0) { tv.wctr[0] = n; tv.wctr[1] = 0; }
}

hipError_t launch_split_level(const Dims& dm, bool full, int lvl, const void* K, const void* V, const void* Q,
                              const float* cosT, const float* sinT, const int32_t* slot_starts,
                              const int32_t* n_slots, const float* kappa, const TreeView& tv, int grid,
                              hipStream_t st);

hipError_t launch_levels(const Dims& dm, bool full, const void* K, const void* V, const void* Q, const float* cosT,
                         const float* sinT, const int32_t* slot_starts, const int32_t* n_slots, const float* kappa,
                         const TreeView& tv, int grid, hipStream_t st) {
  const Dims* dmp = (const Dims*)tv.kargs;
  const TreeView* tvp = (const TreeView*)((const char*)tv.kargs + 512);
  const dim3 lgrid((unsigned)grid);
  hipLaunchKernelGGL(k_level_reset, dim3(1), dim3(64), 0, st, tvp, (int)((int64_t)dm.L * dm.G * dm.J_cap));
  hipLaunchKernelGGL(k_level_first, lgrid, dim3(256), 0, st, dmp, tvp, full ? 1 : 0);
  // depths refined here: LEVELS_MAX; LEVELS_SPARSE at a compression of 64x or
  // more, where the budget-pruned build refines few nodes below that depth and
  // the per-unit kernel ends their chains sooner than a pair of launches per
  // depth would (with less compression the depths stay dense and the rounds
  // are faster).  The complete build takes the same depth, so that both
  // compute every node with the same kernel and round it alike.  Fewer where
  // GRACEKV_LEVELS says so (a knob for tests of the per-unit kernel
  // continuing below the last depth).
  int levels = LEVELS_MAX;
  if (64 * dm.B_total <= (int64_t)dm.L * dm.G * dm.N_ctx) levels = LEVELS_SPARSE;
  if (const char* env = std::getenv("GRACEKV_LEVELS")) {
    const int v = std::atoi(env);
    levels = v < 0 ? 0 : (v < LEVELS_MAX ? v : LEVELS_MAX);
  }
  for (int lvl = 1; lvl <= levels; ++lvl) {
    const hipError_t e = launch_split_level(dm, full, lvl, K, V, Q, cosT, sinT, slot_starts, n_slots, kappa, tv,
                                            grid, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_level, lgrid, dim3(256), 0, st, dmp, tvp, lvl, full ? 1 : 0);
  }
  hipLaunchKernelGGL(k_level_handoff, dim3(1), dim3(256), 0, st, tvp, levels);
  return hipGetLastError();
}

}  // namespace gkv
