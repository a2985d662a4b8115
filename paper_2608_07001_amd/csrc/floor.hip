// Budget-aware singleton floor (App. A.5 Stage I: eq:app_floor_score,
// eq:app_floor_gate, eq:app_floor_cap; App. A.3 split choice with the floor;
// App. C.3 queue initialisation after the floor stage).
//
// Candidates (gracekv_build_trees, once the token values are final):
//   * Rbar_t = mean of R^tok over every (l, g); f_{l,g,t} = max over the
//     tokens tau of C with |tau - t| <= 3 of (1 - c) R_{l,g,tau} + c Rbar_tau,
//     c = 1/2;
//   * per (l, g), the tokens with f >= gamma / N_c (gamma = 1.2) in descending
//     f, ties to the smaller position (a stable LSD radix sort, four 8-bit
//     passes, of the key ~bits(f) over the tokens in position order), kept
//     while the running sum of their R^tok stays <= 0.95 (fp64 running sum);
//     their flags steer the refinement (forced extraction in the tree kernels).
// Realisation (gracekv_select, before the auction), cap = floor(alpha B_base):
//   * a candidate's path: the Add of its unit, then the Split of every
//     ancestor of its leaf {t}; the first list index using each op (atomic
//     minimum) gives both the cost of each (l, g)'s union of paths and each
//     candidate's incremental cost when every earlier candidate of its list is
//     realised;
//   * if the unions cost more than the cap, (l, g) keeps its first
//     max(1, floor(n cap / total)) candidates;
//   * candidates are realised in (l, g) order, each list in order, while their
//     incremental costs fit: up to the first that does not, that is a prefix
//     sum; after it one workgroup walks the rest in order, costing each against
//     the ops executed so far, and realises those that still fit;
//   * B_floor = the cost realised.  The executed ops' effective keys become
//     +inf (their children are exposed with their own keys) and their costs
//     leave the auction, which spends B_base - B_floor.
#include "common.h"

namespace gkv {

constexpr float FLOOR_C = 0.5f;        // cross-head consensus weight (eq:app_floor_score)
constexpr double FLOOR_GAMMA = 1.2;    // quality gate (eq:app_floor_gate)
constexpr double FLOOR_ETA = 0.95;     // cumulative original value of the candidates
constexpr int FLOOR_POOL = 3;          // max-pool half width (width 7)
constexpr int FL_NONE = 0x7fffffff;    // no list index uses the op

static size_t al256f(size_t x) { return (x + 255) & ~(size_t)255; }

FloorView floor_view(void* base, const Dims& dm, int64_t unit_cap, int64_t node_cap) {
  FloorView v;
  const size_t LG = (size_t)dm.L * dm.G, NC = (size_t)dm.N_c;
  char* b = (char*)base;
  size_t o = 0;
  auto take = [&](size_t bytes) { char* p = b ? b + o : nullptr; o += al256f(bytes); return p; };
  v.state = (int64_t*)take(8 * 8);
  v.cnt = (int32_t*)take(LG * 4);
  v.keep = (int32_t*)take(LG * 4);
  v.list = (int32_t*)take(LG * NC * 4);
  v.flag = (uint8_t*)take(LG * NC);
  v.pre_add = (uint8_t*)take((size_t)unit_cap);
  v.pre_sp = (uint8_t*)take((size_t)node_cap);
  v.rbar = (float*)take(NC * 4);
  v.keyA = (uint32_t*)take(LG * NC * 4);
  v.keyB = (uint32_t*)take(LG * NC * 4);
  v.valB = (int32_t*)take(LG * NC * 4);
  v.first_add = (int32_t*)take((size_t)unit_cap * 4);
  v.first_sp = (int32_t*)take((size_t)node_cap * 4);
  v.inc = (int32_t*)take(LG * NC * 4);
  v.lgsum = (int64_t*)take(LG * 8);
  v.bytes = o;
  return v;
}

// ---- candidates -------------------------------------------------------------
__global__ void k_floor_mean(Dims dm, TreeView tv, FloorView fv) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= dm.N_c) return;
  const int LG = dm.L * dm.G;
  float s = 0.f;
  for (int lg = 0; lg < LG; ++lg) s += tv.tok_R[(int64_t)lg * dm.N_c + t];
  fv.rbar[t] = s / (float)LG;
}

// f of every (l, g, t); the sort key ~bits(f) (all ones: below the gate)
__global__ void k_floor_score(Dims dm, TreeView tv, FloorView fv, float gate) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int lg = blockIdx.y;
  if (t >= dm.N_c) return;
  const float* R = tv.tok_R + (int64_t)lg * dm.N_c;
  const int64_t lo = t - FLOOR_POOL > 0 ? t - FLOOR_POOL : 0;
  const int64_t hi = t + FLOOR_POOL < dm.N_c - 1 ? t + FLOOR_POOL : dm.N_c - 1;
  float f = -INFINITY;
  for (int64_t u = lo; u <= hi; ++u) f = fmaxf(f, (1.f - FLOOR_C) * R[u] + FLOOR_C * fv.rbar[u]);
  const int64_t i = (int64_t)lg * dm.N_c + t;
  fv.keyB[i] = f >= gate ? ~__float_as_uint(f) : 0xFFFFFFFFu;
  fv.flag[i] = 0;
}

constexpr int FS_T = 256;

// lanes below this one
__device__ __forceinline__ uint64_t lanes_below(int lane) { return lane == 0 ? 0ull : (~0ull >> (64 - lane)); }

// One stable LSD radix pass (8 bits at `shift`) of m (key, value) pairs by one
// workgroup: digit histogram, exclusive starts, then chunks of 256 in order,
// each element placed after the earlier elements of its digit (earlier waves,
// then earlier lanes of its wave, found by matching the digit over 8 ballots).
__device__ void floor_radix_pass(const uint32_t* kin, const int32_t* vin, uint32_t* kout, int32_t* vout, int m,
                                 int shift, int* start, int (*wcnt)[256]) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  start[tid] = 0;
  for (int w = 0; w < 4; ++w) wcnt[w][tid] = 0;
  __syncthreads();
  for (int i = tid; i < m; i += FS_T) atomicAdd(&start[(kin[i] >> shift) & 255u], 1);
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int d = 0; d < 256; ++d) { const int c = start[d]; start[d] = acc; acc += c; }
  }
  __syncthreads();
  for (int c0 = 0; c0 < m; c0 += FS_T) {
    const int i = c0 + tid;
    const bool valid = i < m;
    const uint32_t key = valid ? kin[i] : 0u;
    const int32_t val = valid ? vin[i] : 0;
    const int d = (int)((key >> shift) & 255u);
    uint64_t mask = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t bb = __ballot(valid && ((d >> b) & 1));
      mask &= ((d >> b) & 1) ? bb : ~bb;
    }
    const int rank = __popcll(mask & lanes_below(lane));
    if (valid && rank == 0) wcnt[wave][d] = __popcll(mask);
    __syncthreads();
    if (valid) {
      int off = start[d] + rank;
      for (int w = 0; w < wave; ++w) off += wcnt[w][d];
      kout[off] = key;
      vout[off] = val;
    }
    __syncthreads();
    start[tid] += wcnt[0][tid] + wcnt[1][tid] + wcnt[2][tid] + wcnt[3][tid];
    for (int w = 0; w < 4; ++w) wcnt[w][tid] = 0;
    __syncthreads();
  }
}

// One workgroup per (l, g): the gated tokens in position order, sorted by key,
// then the list cut where the running sum of R^tok first exceeds 0.95.
__global__ __launch_bounds__(FS_T) void k_floor_sort(Dims dm, TreeView tv, FloorView fv) {
  const int lg = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t row = (int64_t)lg * dm.N_c;
  const int N = (int)dm.N_c;
  __shared__ int start[256];
  __shared__ int wcnt[4][256];
  __shared__ int wtot[4];
  __shared__ double dtot[4];
  __shared__ int carry_i, found;
  __shared__ double carry_d;
  uint32_t* kA = fv.keyA + row;
  uint32_t* kB = fv.keyB + row;
  int32_t* vA = fv.list + row;
  int32_t* vB = fv.valB + row;
  // compaction of the gated tokens (position order) into A
  if (tid == 0) carry_i = 0;
  __syncthreads();
  for (int c0 = 0; c0 < N; c0 += FS_T) {
    const int t = c0 + tid;
    const uint32_t key = t < N ? kB[t] : 0xFFFFFFFFu;
    const bool on = key != 0xFFFFFFFFu;
    const uint64_t m = __ballot(on);
    if (lane == 0) wtot[wave] = __popcll(m);
    __syncthreads();
    int off = carry_i + __popcll(m & lanes_below(lane));
    for (int w = 0; w < wave; ++w) off += wtot[w];
    if (on) { kA[off] = key; vA[off] = t; }
    __syncthreads();
    if (tid == 0) carry_i += wtot[0] + wtot[1] + wtot[2] + wtot[3];
    __syncthreads();
  }
  const int m0 = carry_i;
  // four stable passes: A -> B -> A -> B -> A
  floor_radix_pass(kA, vA, kB, vB, m0, 0, start, wcnt);
  floor_radix_pass(kB, vB, kA, vA, m0, 8, start, wcnt);
  floor_radix_pass(kA, vA, kB, vB, m0, 16, start, wcnt);
  floor_radix_pass(kB, vB, kA, vA, m0, 24, start, wcnt);
  // the list stops before the first token whose R^tok takes the running sum above eta
  if (tid == 0) { carry_d = 0.0; found = m0; }
  __syncthreads();
  const float* R = tv.tok_R + row;
  for (int c0 = 0; c0 < m0; c0 += FS_T) {
    const int i = c0 + tid;
    double x = i < m0 ? (double)R[vA[i]] : 0.0;
    // inclusive scan within the wave, then over the waves
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const double y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) dtot[wave] = x;
    __syncthreads();
    double s = carry_d;
    for (int w = 0; w < wave; ++w) s += dtot[w];
    s += x;
    const bool over = i < m0 && s > FLOOR_ETA;
    if (over) atomicMin(&found, i);
    __syncthreads();
    if (tid == 0) carry_d += dtot[0] + dtot[1] + dtot[2] + dtot[3];
    __syncthreads();
    if (found < m0) break;
  }
  const int m = found;
  for (int i = tid; i < m; i += FS_T) fv.flag[row + vA[i]] = 1;
  if (tid == 0) fv.cnt[lg] = m;
}

hipError_t launch_floor_candidates(const Dims& dm, const TreeView& tv, const FloorView& fv, hipStream_t st) {
  const int LG = dm.L * dm.G;
  const unsigned nb = (unsigned)((dm.N_c + 255) / 256);
  hipLaunchKernelGGL(k_floor_mean, dim3(nb), dim3(256), 0, st, dm, tv, fv);
  const float gate = (float)(FLOOR_GAMMA / (double)dm.N_c);
  hipLaunchKernelGGL(k_floor_score, dim3(nb, LG), dim3(256), 0, st, dm, tv, fv, gate);
  hipLaunchKernelGGL(k_floor_sort, dim3(LG), dim3(FS_T), 0, st, dm, tv, fv);
  return hipGetLastError();
}

// ---- realisation --------------------------------------------------------------
// The ops on the path of candidate t of (l, g): the Add of its unit, then the
// Split of every ancestor of the leaf {t}, root first; fn(is_split, index
// (unit, or node slot), cost).  Returns the unit.
template <typename F>
__device__ int64_t floor_path(const Dims& dm, const TreeView& tv, int lg, int t, int J, F fn) {
  int lo = 0, hi = J - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tv.slots[mid] <= t) lo = mid; else hi = mid - 1;
  }
  const int64_t u = (int64_t)lg * dm.J_cap + lo;
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)tv.slots[lo];
  fn(false, u, 1);
  int node = 0;
  for (int step = 0; step < NODE_MAX; ++step) {
    const int64_t s = base + node;
    const int nch = tv.node_nch[s];
    if (nch == 0) break;
    fn(true, s, nch - 1);
    const int c0 = tv.node_child[s];
    int next = c0;
    for (int k = 0; k < nch; ++k) {
      const int64_t sc = base + c0 + k;
      const int a = tv.node_a[sc];
      if (a <= t && t < a + tv.node_n[sc]) { next = c0 + k; break; }
    }
    node = next;
  }
  return u;
}

__global__ void k_floor_reset(Dims dm, FloorView fv, int64_t unit_cap, int64_t node_cap) {
  const int64_t LGN = (int64_t)dm.L * dm.G * dm.N_c;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < node_cap; i += stride) {
    fv.first_sp[i] = FL_NONE;
    fv.pre_sp[i] = 0;
    if (i < unit_cap) { fv.first_add[i] = FL_NONE; fv.pre_add[i] = 0; }
    if (i < LGN) fv.inc[i] = 0;
    if (i < dm.L * dm.G) fv.lgsum[i] = 0;
    if (i < 8) fv.state[i] = i == 4 ? dm.L * dm.G : 0;   // no failure point yet
  }
}

// first list index using each op, over the initial lists
__global__ void k_floor_first(Dims dm, TreeView tv, FloorView fv) {
  const int lg = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= fv.cnt[lg]) return;
  const int J = *tv.nslots;
  const int t = fv.list[(int64_t)lg * dm.N_c + i];
  floor_path(dm, tv, lg, t, J, [&](bool sp, int64_t x, int) {
    atomicMin(sp ? &fv.first_sp[x] : &fv.first_add[x], i);
  });
}

// cost of each (l, g)'s union of paths, and each candidate's incremental cost
__global__ void k_floor_costs(Dims dm, TreeView tv, FloorView fv, int64_t unit_cap, int64_t node_cap) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < node_cap + unit_cap; x += stride) {
    int first, cost, lg;
    if (x < node_cap) {
      first = fv.first_sp[x];
      if (first == FL_NONE) continue;
      cost = tv.node_nch[x] - 1;
      lg = (int)(x / (2 * dm.N_c));
    } else {
      const int64_t u = x - node_cap;
      first = fv.first_add[u];
      if (first == FL_NONE) continue;
      cost = 1;
      lg = (int)(u / dm.J_cap);
    }
    atomicAdd((unsigned long long*)&fv.lgsum[lg], (unsigned long long)cost);
    atomicAdd(&fv.inc[(int64_t)lg * dm.N_c + first], cost);
  }
}

// the proportional reduction (eq:app_floor_cap); then lgsum = the kept
// candidates' incremental costs of each (l, g)
__global__ void k_floor_plan(Dims dm, FloorView fv) {
  const int LG = dm.L * dm.G;
  __shared__ unsigned long long tot;
  if (threadIdx.x == 0) tot = 0;
  __syncthreads();
  unsigned long long s = 0;
  for (int lg = threadIdx.x; lg < LG; lg += blockDim.x) s += (unsigned long long)fv.lgsum[lg];
  atomicAdd(&tot, s);
  __syncthreads();
  const int64_t total = (int64_t)tot, cap = dm.floor_cap;
  const bool reduced = total > cap;
  for (int lg = threadIdx.x; lg < LG; lg += blockDim.x) {
    const int n = fv.cnt[lg];
    int k = n;
    if (reduced && n > 0) {
      const int64_t q = (int64_t)n * cap / total;
      k = (int)(q > 1 ? q : 1);
    }
    fv.keep[lg] = k;
  }
  if (threadIdx.x == 0) { fv.state[1] = cap; fv.state[2] = total; fv.state[3] = reduced ? 1 : 0; }
}

__global__ __launch_bounds__(256) void k_floor_keptsum(Dims dm, FloorView fv) {
  const int lg = blockIdx.x;
  __shared__ unsigned long long acc;
  if (threadIdx.x == 0) acc = 0;
  __syncthreads();
  unsigned long long s = 0;
  const int k = fv.keep[lg];
  for (int i = threadIdx.x; i < k; i += 256) s += (unsigned long long)fv.inc[(int64_t)lg * dm.N_c + i];
  atomicAdd(&acc, s);
  __syncthreads();
  if (threadIdx.x == 0) fv.lgsum[lg] = (int64_t)acc;
}

// the first candidate (in (l, g) order, each list in order) whose incremental
// cost does not fit: state[4] = its (l, g) (LG: none), state[5] = its index,
// state[6] = the cost realised before it
__global__ __launch_bounds__(256) void k_floor_fail(Dims dm, FloorView fv) {
  const int LG = dm.L * dm.G;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  __shared__ int lgF;
  __shared__ long long before;
  // (a candidate is always found in the failing (l, g): its kept costs exceed the rest)
  __shared__ long long wsum[4];
  __shared__ long long carry;
  __shared__ int iF;
  const int64_t cap = dm.floor_cap;
  if (tid == 0) {
    long long acc = 0;
    int f = LG;
    for (int lg = 0; lg < LG; ++lg) {
      if (acc + fv.lgsum[lg] > cap) { f = lg; break; }
      acc += fv.lgsum[lg];
    }
    lgF = f;
    before = acc;
    carry = acc;
    iF = 0x7fffffff;
  }
  __syncthreads();
  if (lgF == LG) {
    if (tid == 0) { fv.state[0] = before; fv.state[4] = LG; fv.state[5] = 0; fv.state[6] = before; }
    return;
  }
  const int k = fv.keep[lgF];
  const int32_t* inc = fv.inc + (int64_t)lgF * dm.N_c;
  for (int c0 = 0; c0 < k; c0 += 256) {
    const int i = c0 + tid;
    long long x = i < k ? inc[i] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const long long y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    long long s = carry;
    for (int w = 0; w < wave; ++w) s += wsum[w];
    s += x;
    if (i < k && s > cap) atomicMin(&iF, i);
    __syncthreads();
    if (i == iF) {                            // the cost realised before the failing candidate
      const long long acc = s - inc[i];
      fv.state[4] = lgF;
      fv.state[5] = iF;
      fv.state[6] = acc;
      fv.state[0] = acc;
    }
    if (tid == 0) carry += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
    if (iF != 0x7fffffff) break;
  }
}

// the ops of the candidates realised before the failure point
__global__ void k_floor_mark(Dims dm, FloorView fv, int64_t unit_cap, int64_t node_cap) {
  const int64_t lgF = fv.state[4], iF = fv.state[5];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < node_cap + unit_cap; x += stride) {
    int first, lg;
    if (x < node_cap) { first = fv.first_sp[x]; lg = (int)(x / (2 * dm.N_c)); }
    else { first = fv.first_add[x - node_cap]; lg = (int)((x - node_cap) / dm.J_cap); }
    if (first == FL_NONE || first >= fv.keep[lg]) continue;
    if (lg < lgF || (lg == lgF && first < iF)) {
      if (x < node_cap) fv.pre_sp[x] = 1; else fv.pre_add[x - node_cap] = 1;
    }
  }
}

// path cost of the candidates after the failure point against the ops
// executed so far, and their units
__global__ void k_floor_c0(Dims dm, TreeView tv, FloorView fv) {
  const int lg = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  const int64_t lgF = fv.state[4], iF = fv.state[5];
  if (lg < lgF || i >= fv.keep[lg] || (lg == lgF && i <= iF)) return;
  const int J = *tv.nslots;
  const int64_t at = (int64_t)lg * dm.N_c + i;
  int c = 0;
  const int64_t u = floor_path(dm, tv, lg, fv.list[at], J, [&](bool sp, int64_t x, int cost) {
    if (!(sp ? fv.pre_sp[x] : fv.pre_add[x])) c += cost;
  });
  fv.keyB[at] = (uint32_t)c;
  fv.valB[at] = (int32_t)u;
}

// After the failure point, in order: a candidate is realised iff its cost
// against the ops executed so far fits the rest of the cap.  A candidate whose
// cost before the tail exceeds the rest can only fit once a tail realisation
// shares its unit, so only those are walked again.
constexpr int FT_UNITS = 256;
__global__ __launch_bounds__(256) void k_floor_tail(Dims dm, TreeView tv, FloorView fv) {
  const int LG = dm.L * dm.G;
  const int tid = threadIdx.x;
  const int64_t lgF = fv.state[4];
  if (lgF >= LG) return;
  const int J = *tv.nslots;
  __shared__ long long rem;
  __shared__ int win, win_c, nunits;
  __shared__ int64_t units[FT_UNITS];
  if (tid == 0) { rem = dm.floor_cap - fv.state[6]; nunits = 0; }
  __syncthreads();
  for (int lg = (int)lgF; lg < LG; ++lg) {
    const int k = fv.keep[lg];
    int pos = lg == lgF ? (int)fv.state[5] + 1 : 0;
    while (pos < k && rem > 0) {
      const int i = pos + tid;
      int c = -1;
      if (i < k) {
        const int64_t at = (int64_t)lg * dm.N_c + i;
        c = (int)fv.keyB[at];
        bool walk = c > 0 && c <= rem;
        if (!walk && c > rem) {
          if (nunits > FT_UNITS) {
            walk = true;                      // the unit list overflowed: walk every candidate
          } else {
            const int64_t u = fv.valB[at];
            for (int q = 0; q < nunits; ++q) walk |= units[q] == u;
          }
        }
        if (walk) {
          c = 0;
          floor_path(dm, tv, lg, fv.list[at], J, [&](bool sp, int64_t x, int cost) {
            if (!(sp ? fv.pre_sp[x] : fv.pre_add[x])) c += cost;
          });
        }
      }
      if (tid == 0) win = 0x7fffffff;
      __syncthreads();
      if (i < k && c > 0 && c <= rem) atomicMin(&win, tid);
      __syncthreads();
      const int w = win;
      if (w == 0x7fffffff) {
        pos += 256;
        __syncthreads();
        continue;
      }
      if (tid == w) {
        const int64_t u = floor_path(dm, tv, lg, fv.list[(int64_t)lg * dm.N_c + i], J,
                                     [&](bool sp, int64_t x, int) {
                                       if (sp) fv.pre_sp[x] = 1; else fv.pre_add[x] = 1;
                                     });
        rem -= c;
        if (nunits < FT_UNITS) units[nunits] = u;
        nunits += 1;
        if (nunits > FT_UNITS) nunits = FT_UNITS + 1;   // the list is full: every candidate is walked
      }
      // the marks, visible to the workgroup's later walks
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __syncthreads();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      pos = pos + w + 1;
    }
  }
  if (tid == 0) fv.state[0] = dm.floor_cap - rem;
}

// effective keys with the floor's executions: +inf for an executed op, its
// children exposed with their own keys
__global__ void k_floor_rekey(Dims dm, TreeView tv, FloorView fv) {
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= (int64_t)dm.L * dm.G * dm.J_cap) return;
  const int lg = (int)(u / dm.J_cap), j = (int)(u % dm.J_cap);
  const int J = *tv.nslots;
  if (j >= J) return;
  const int nn = tv.unit_nn[u];
  if (nn < 1) return;
  const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * (int64_t)tv.slots[j];
  const uint64_t INF = ~0ull;
  const uint64_t Ea = fv.pre_add[u] ? INF : op_key(tv.add_U[u], ord * 256u);
  tv.add_E[u] = Ea;
  for (int i = 0; i < nn; ++i) {
    const int64_t s = base + i;
    if (tv.node_nch[s] == 0) continue;
    const int par = tv.node_parent[s];
    const uint64_t Ep = par < 0 ? Ea : tv.sp_E[base + par];
    const uint64_t k = op_key(tv.sp_U[s], ord * 256u + 1u + (uint32_t)i);
    tv.sp_E[s] = fv.pre_sp[s] ? INF : (k < Ep ? k : Ep);
  }
}

hipError_t launch_floor_realise(const Dims& dm, const TreeView& tv, const FloorView& fv, hipStream_t st) {
  const int LG = dm.L * dm.G;
  const int64_t unit_cap = (int64_t)LG * dm.J_cap, node_cap = (int64_t)LG * 2 * dm.N_c;
  const unsigned nb = (unsigned)((dm.N_c + 255) / 256);
  hipLaunchKernelGGL(k_floor_reset, dim3(2048), dim3(256), 0, st, dm, fv, unit_cap, node_cap);
  hipLaunchKernelGGL(k_floor_first, dim3(nb, LG), dim3(256), 0, st, dm, tv, fv);
  hipLaunchKernelGGL(k_floor_costs, dim3(2048), dim3(256), 0, st, dm, tv, fv, unit_cap, node_cap);
  hipLaunchKernelGGL(k_floor_plan, dim3(1), dim3(256), 0, st, dm, fv);
  hipLaunchKernelGGL(k_floor_keptsum, dim3(LG), dim3(256), 0, st, dm, fv);
  hipLaunchKernelGGL(k_floor_fail, dim3(1), dim3(256), 0, st, dm, fv);
  hipLaunchKernelGGL(k_floor_mark, dim3(2048), dim3(256), 0, st, dm, fv, unit_cap, node_cap);
  hipLaunchKernelGGL(k_floor_c0, dim3(nb, LG), dim3(256), 0, st, dm, tv, fv);
  hipLaunchKernelGGL(k_floor_tail, dim3(1), dim3(256), 0, st, dm, tv, fv);
  hipLaunchKernelGGL(k_floor_rekey, dim3((unsigned)((unit_cap + 127) / 128)), dim3(128), 0, st, dm, tv, fv);
  return hipGetLastError();
}

}  // namespace gkv
