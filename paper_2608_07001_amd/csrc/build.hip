// Prototype-tree refinement of the units that need it.
//
// Implements App. A.3: RoPE-consistent key prototype eq:app_rope_prototype,
// value prototype eq:app_value_prototype, effective multiplicity
// eq:app_effective_multiplicity, distortion eq:app_original_attention_stats ..
// eq:app_node_and_drop_distortion, recursive refinement eq:app_binary_split ..
// eq:app_split_choice.  The root of every unit, the token values R_t and the
// probe masses A_t come from the root kernel; this kernel resumes from the
// node table.
//
// A mark kernel lists the units with a node to refine (all of them, or only
// those whose creating operation reaches the auction bound theta); one
// workgroup per CU then drains the list.  Per unit (n <= 128 tokens, 512
// threads):
//   * staging: k° = RoPE^{-1}(k) of every token (fp32), V^T (bf16 or fp32),
//     R_t, A_t, curvature, ||k_t|| go to LDS; each wave keeps the quarter rows
//     of its 16 distortion probes in registers;
//   * per node [a, b) in BFS order: the candidate children are prefixes
//     [a, x) and suffixes [x, b) (binary cuts and the extraction sides).
//       - prototype sums: one half of the workgroup sweeps k°, R v, v left to
//         right, the other right to left, and reads the child sums off at the
//         cuts;
//       - child prototypes (coherence, multiplicity, representative position,
//         k~, v~), then z_{q,c} = m_eff exp(q.k~ / sqrt(d) - m_q) for every
//         probe and child on the matrix cores;
//       - M_q(child) = sum_t e_{q,t} v_t on the matrix cores: wave (probe tile,
//         direction) recomputes e for a 16-token block (transposed logits, so e
//         is already the B operand), accumulates M^T = V^T E^T piece by piece
//         between cuts (e split into three bf16 parts: exact products), and at
//         each cut turns the running sums into D_q for that child;
//     then the fp32 scores decide (binary form wins ties, smaller cut wins
//     ties) and the children are appended;
//   * the node table is written back.
#include "common.h"

namespace gkv {

constexpr int BT = 512;          // threads per workgroup
constexpr int NWV = BT / 64;     // waves: (probe tile w % 4, direction w / 4)
constexpr int GT = 256;          // threads per direction group in the prototype sums
constexpr int CM = CAND_MAX;     // children per direction: up to 17 cuts + one extraction side
constexpr int CC = 2 * CM;       // child slots: prefix side [0, CM), suffix side [CM, 2 CM)

template <typename T, int D>
struct RefLds {
  static constexpr bool BF = sizeof(T) == 2;
  static constexpr int LDV = BF ? NMAX + 8 : NMAX + 4;   // V^T row stride
  static constexpr int KTS = D + 4;                       // k~ row stride
  static constexpr int oKo = 0;                           // k° [NMAX][D] fp32
  static constexpr int oVt = oKo + NMAX * D * 4;          // V^T [D][LDV]
  static constexpr int oR = oVt + D * LDV * (int)sizeof(T);
  static constexpr int oA = oR + NMAX * 4;
  static constexpr int oKap = oA + NMAX * 4;
  static constexpr int oKn = oKap + NMAX * 4;
  static constexpr int oMq = oKn + NMAX * 4;              // [WMAX] m_q
  static constexpr int oZc = oMq + WMAX * 4;              // [WMAX] Z_q(C)
  static constexpr int oNa = oZc + WMAX * 4;              // node table, 256 entries each
  static constexpr int oNn = oNa + 256 * 4;
  static constexpr int oNc = oNn + 256 * 4;
  static constexpr int oNp = oNc + 256 * 4;
  static constexpr int oNcut = oNp + 256 * 4;
  static constexpr int oND = oNcut + 256 * 4;
  static constexpr int oNR = oND + 256 * 4;
  static constexpr int oNU = oNR + 256 * 4;
  static constexpr int oNE = oNU + 256 * 4;               // uint64
  static constexpr int oNch = oNE + 256 * 8;              // uint8
  static constexpr int oNk = oNch + 256;
  static constexpr int oKt = oNk + 256;                   // [CC][KTS] mean k° -> k~; then per-wave D sums [CC][4]
  static constexpr int oVv = oKt + CC * KTS * 4;          // [CC][D] v~
  static constexpr int oZt = oVv + CC * D * 4;            // [CC][WMAX] z_{q,c}
  static constexpr int oCs = oZt + CC * WMAX * 4;         // [5][CC] n, sum R, mean ||k||, m_eff, D
  static constexpr int oX = oCs + 5 * CC * 4;             // cut lists and metadata
  static constexpr int oFlag = oX + 256 * 4;
  static constexpr int oFl = oFlag + NMAX * 4;            // [NMAX] singleton-floor candidate flags
  static constexpr int bytes = oFl + NMAX;
};

int build_lds_bytes(const Dims& dm) {
  if (dm.dtype == GRACEKV_BF16) return dm.d == 128 ? RefLds<uint16_t, 128>::bytes : RefLds<uint16_t, 64>::bytes;
  return dm.d == 128 ? RefLds<float, 128>::bytes : RefLds<float, 64>::bytes;
}

template <typename T, int D>
struct Ref {
  using Lay = RefLds<T, D>;
  char* s;
  float* Ko; T* Vt; float* R; float* A; float* Kap; float* Kn; float* Mq; float* Zc;
  int* na; int* nn; int* nc; int* np; int* ncut; float* nD; float* nR; float* nU; uint64_t* nE;
  uint8_t* nch; uint8_t* nk;
  float* Kt; float* Con; float* Vv; float* Zt; float* cs; int* xi; int* flag; uint8_t* fl;
  __device__ Ref(char* base) : s(base) {
    Ko = (float*)(s + Lay::oKo); Vt = (T*)(s + Lay::oVt); R = (float*)(s + Lay::oR); A = (float*)(s + Lay::oA);
    Kap = (float*)(s + Lay::oKap); Kn = (float*)(s + Lay::oKn); Mq = (float*)(s + Lay::oMq);
    Zc = (float*)(s + Lay::oZc);
    na = (int*)(s + Lay::oNa); nn = (int*)(s + Lay::oNn); nc = (int*)(s + Lay::oNc); np = (int*)(s + Lay::oNp);
    ncut = (int*)(s + Lay::oNcut); nD = (float*)(s + Lay::oND); nR = (float*)(s + Lay::oNR);
    nU = (float*)(s + Lay::oNU); nE = (uint64_t*)(s + Lay::oNE);
    nch = (uint8_t*)(s + Lay::oNch); nk = (uint8_t*)(s + Lay::oNk);
    Kt = (float*)(s + Lay::oKt); Con = Kt; Vv = (float*)(s + Lay::oVv); Zt = (float*)(s + Lay::oZt);
    cs = (float*)(s + Lay::oCs); xi = (int*)(s + Lay::oX); flag = (int*)(s + Lay::oFlag);
    fl = (uint8_t*)(s + Lay::oFl);
  }
  __device__ float* crow(int row) { return cs + row * CC; }
};

// x = hi + mid + lo exactly, each a bf16 (hi: top 8 significant bits by
// truncation, mid: the next 8, lo: the rest), packed two per 32-bit word as
// the matrix-core operands want them
__device__ __forceinline__ void split3x4(const float* x, u32x2& hi, u32x2& mid, u32x2& lo) {
  uint32_t h[4], m[4], l[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    h[r] = __float_as_uint(x[r]) & 0xffff0000u;
    const float r1 = x[r] - __uint_as_float(h[r]);
    m[r] = __float_as_uint(r1) & 0xffff0000u;
    l[r] = __float_as_uint(r1 - __uint_as_float(m[r]));
  }
#define GKV_HI2(a, b) __builtin_amdgcn_perm((b), (a), 0x07060302u)
  hi.x = GKV_HI2(h[0], h[1]); hi.y = GKV_HI2(h[2], h[3]);
  mid.x = GKV_HI2(m[0], m[1]); mid.y = GKV_HI2(m[2], m[3]);
  lo.x = GKV_HI2(l[0], l[1]); lo.y = GKV_HI2(l[2], l[3]);
#undef GKV_HI2
}
__device__ __forceinline__ s16x4 as_op(u32x2 v) { return __builtin_bit_cast(s16x4, v); }

// ---------------------------------------------------------------------------
// Prototype sums of both directions at once.  Group 0 reads the prefix
// children [a, XL[c]) off a left-to-right sweep, group 1 the suffix children
// [XR[c], b) off a right-to-left sweep.  Child slot gc = g * CM + c gets
// mean k° (Kt), v~ (Vv), n, sum R and mean ||k|| (cs rows 0..2).
template <typename T, int D>
__device__ void proto_sums(Ref<T, D>& U, const Dims& dm, int a, int b, const int* XL, int nl, const int* XR,
                           int nr) {
  using Lay = RefLds<T, D>;
  const int tid = threadIdx.x;
  const int g = tid / GT, lt = tid % GT;
  const bool prefix = g == 0;
  const int* xs = prefix ? XL : XR;
  const int nx = prefix ? nl : nr;
  if (lt >= 2 * D || nx == 0) return;
  const bool kside = lt < D;
  const int i = kside ? lt : lt - D;
  float s0 = 0.f, s1 = 0.f, sr = 0.f, skn = 0.f;
  int t = prefix ? a : b - 1;                 // next token of the sweep
  for (int k = 0; k < nx; ++k) {
    const int c = prefix ? k : nx - 1 - k;
    const int x = xs[c];
    // tokens up to the read-off: prefix [t, x), suffix down to x (inclusive)
    const int cntk = prefix ? x - t : t - x + 1;
    const int step = prefix ? 1 : -1;
    if (kside) {
      int u = 0;
      for (; u + 4 <= cntk; u += 4) {
        float f[4], kk[4], rr[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int tt = t + step * (u + v);
          f[v] = U.Ko[tt * D + i]; kk[v] = U.Kn[tt]; rr[v] = U.R[tt];
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) { s0 += f[v]; skn += kk[v]; sr += rr[v]; }
      }
      for (; u < cntk; ++u) {
        const int tt = t + step * u;
        s0 += U.Ko[tt * D + i]; skn += U.Kn[tt]; sr += U.R[tt];
      }
    } else {
      int u = 0;
      for (; u + 4 <= cntk; u += 4) {
        float f[4], rr[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int tt = t + step * (u + v);
          f[v] = ldf(U.Vt, i * Lay::LDV + tt); rr[v] = U.R[tt];
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) { s0 += rr[v] * f[v]; s1 += f[v]; sr += rr[v]; }
      }
      for (; u < cntk; ++u) {
        const int tt = t + step * u;
        const float f = ldf(U.Vt, i * Lay::LDV + tt), rr = U.R[tt];
        s0 += rr * f; s1 += f; sr += rr;
      }
    }
    t += step * cntk;
    const int nch = prefix ? x - a : b - x;
    const int gc = g * CM + c;
    if (nch >= 2) {
      const float inv = 1.0f / (float)nch;
      if (kside) {
        U.Kt[gc * Lay::KTS + i] = s0 * inv;
      } else {
        const float beta = dm.beta_frac * sr * inv;
        U.Vv[gc * D + i] = (s0 + beta * s1) / (sr + (float)nch * beta + dm.eps);
      }
    }
    if (lt == 0) {
      U.crow(0)[gc] = (float)nch;
      U.crow(1)[gc] = sr;
      U.crow(2)[gc] = skn / (float)nch;
    }
  }
}

// Child prototypes: coherence, multiplicity, representative position and
// k~ = RoPE(mean k°, p) in place (one wave per child).
template <typename T, int D>
__device__ void proto_keys(Ref<T, D>& U, const Dims& dm, int64_t a0, int a, int b, const int* XL, int nl,
                           const int* XR, int nr, const float* __restrict__ cosT, const float* __restrict__ sinT) {
  using Lay = RefLds<T, D>;
  constexpr int H2 = D / 2;
  constexpr int KPW = (CC + NWV - 1) / NWV;   // children per wave
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = lane < H2 ? lane : 0;         // the lane's rotation pair (i, i + H2)
  // rotation rows of the wave's children, all loads in flight together
  float cc[KPW], sn[KPW];
#pragma unroll
  for (int m = 0; m < KPW; ++m) {
    const int k = wave + NWV * m;
    cc[m] = 1.f;
    sn[m] = 0.f;
    if (k < nl + nr) {
      const bool pre = k < nl;
      const int c = pre ? k : k - nl;
      const int x0 = pre ? a : XR[c];
      const int x1 = pre ? XL[c] : b;
      const int64_t p = round_half_even_mid((int)(a0 + x0), (int)(a0 + x1));
      cc[m] = cosT[p * H2 + i];
      sn[m] = sinT[p * H2 + i];
    }
  }
#pragma unroll
  for (int m = 0; m < KPW; ++m) {
    const int k = wave + NWV * m;
    if (k >= nl + nr) break;
    const bool pre = k < nl;
    const int c = pre ? k : k - nl;
    const int gc = pre ? c : CM + c;
    const int nch = (int)U.crow(0)[gc];
    if (nch < 2) continue;
    float* kt = U.Kt + gc * Lay::KTS;
    float ss = 0.f;
    for (int d = lane; d < D; d += 64) ss += kt[d] * kt[d];
    ss = wave_sum_dpp(ss);
    const float coh = sqrtf(ss) / (U.crow(2)[gc] + dm.eps);
    const float me = fminf(fmaxf((float)nch * coh * coh, 1.0f), (float)nch);
    if (lane == 0) U.crow(3)[gc] = me;
    if (lane < H2) {
      const float m1 = kt[i], m2 = kt[i + H2];
      kt[i] = m1 * cc[m] - m2 * sn[m];
      kt[i + H2] = m2 * cc[m] + m1 * sn[m];
    }
  }
}

// z_{q,c} = m_eff(c) exp(q . k~_c / sqrt(d) - m_q) for the wave's probe tile
// and child tiles; A = probe rows (registers), B = k~ rows (fp32, split in three
// bf16 parts for the bf16 path).
template <typename T, int D, int QW>
__device__ void proto_attention(Ref<T, D>& U, const Dims& dm, int nl, int nr, const uint32_t* qreg, int pt,
                                float scale) {
  using Lay = RefLds<T, D>;
  constexpr bool BF = Lay::BF;
  constexpr int QE = D / 4;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, i16 = lane & 15, g4 = lane >> 4;
  if (16 * pt >= dm.W) return;
  for (int ct = wave >> 2; ct < (CC + 15) / 16; ct += 2) {
    const int gc = 16 * ct + i16;
    const int gcc = gc < CC ? gc : 0;
    const bool live = gc < CC && ((gc < CM && gc < nl) || (gc >= CM && gc - CM < nr));
    const bool cok = live && U.crow(0)[gcc] >= 2.f;
    if (!__any(cok)) continue;                // the tile holds no child to score (wave-uniform)
    const float* kt = U.Kt + gcc * Lay::KTS + QE * g4;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (BF) {
#pragma unroll
      for (int s = 0; s < QE / 4; ++s) {
        float x[4];
        const float4 v = *(const float4*)(kt + 4 * s);
        x[0] = cok ? v.x : 0.f; x[1] = cok ? v.y : 0.f; x[2] = cok ? v.z : 0.f; x[3] = cok ? v.w : 0.f;
        u32x2 h, m, l;
        split3x4(x, h, m, l);
        const s16x4 qa = pk4(qreg[2 * s], qreg[2 * s + 1]);
        acc = mfma_bf16_16x16x16(qa, as_op(l), acc);
        acc = mfma_bf16_16x16x16(qa, as_op(m), acc);
        acc = mfma_bf16_16x16x16(qa, as_op(h), acc);
      }
    } else {
#pragma unroll
      for (int s = 0; s < QE; ++s) acc = mfma_f32_16x16x4(__uint_as_float(qreg[s]), cok ? kt[s] : 0.f, acc);
    }
    // lane holds probes 16 pt + 4 g4 + r of child gc
    if (cok) {
      const float me = U.crow(3)[gc];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = 16 * pt + 4 * g4 + r;
        if (q < dm.W) U.Zt[gc * WMAX + q] = me * fexp(acc[r] * scale - U.Mq[q]);
      }
    }
  }
}

// the lane's key quarter row of block blk (unit-local token 16 blk + i16,
// clamped to the unit)
template <typename T, int D, int QW>
__device__ __forceinline__ void block_k(const T* __restrict__ Kp, int n, int blk, uint32_t* kreg) {
  constexpr int QE = D / 4;
  const int lane = threadIdx.x & 63, i16 = lane & 15, g4 = lane >> 4;
  int tr = 16 * blk + i16;
  tr = tr < n ? tr : n - 1;
  const uint4* k4 = (const uint4*)(Kp + (int64_t)tr * D + QE * g4);
#pragma unroll
  for (int h = 0; h < QW / 4; ++h) {
    const uint4 v = k4[h];
    kreg[4 * h] = v.x; kreg[4 * h + 1] = v.y; kreg[4 * h + 2] = v.z; kreg[4 * h + 3] = v.w;
  }
}

// e_{q,t} for the 16 tokens of block blk and the lane's probe: transposed
// logits, lane holds tokens 16 blk + 4 g4 + r; e = 2^(l sc2 - mq2) with the
// logit scale and the probe shift in base-2 units.  The lane's key and probe
// registers cover dims QE g4 .. QE g4 + QE - 1, eight per 16x16x32 step.
template <typename T, int D, int QW>
__device__ __forceinline__ void block_e(const uint32_t* kreg, int n, int blk, const uint32_t* qreg, float mq2,
                                        bool pok, float sc2, float* ev) {
  constexpr bool BF = sizeof(T) == 2;
  constexpr int QE = D / 4;
  const int lane = threadIdx.x & 63, g4 = lane >> 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if constexpr (BF) {
#pragma unroll
    for (int s = 0; s < QE / 8; ++s)
      acc = mfma_bf16_16x16x32(pk8(make_uint4(kreg[4 * s], kreg[4 * s + 1], kreg[4 * s + 2], kreg[4 * s + 3])),
                               pk8(make_uint4(qreg[4 * s], qreg[4 * s + 1], qreg[4 * s + 2], qreg[4 * s + 3])), acc);
  } else {
#pragma unroll
    for (int s = 0; s < QE; ++s) acc = mfma_f32_16x16x4(__uint_as_float(kreg[s]), __uint_as_float(qreg[s]), acc);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int t = 16 * blk + 4 * g4 + r;
    ev[r] = __builtin_amdgcn_exp2f((pok && t < n) ? acc[r] * sc2 - mq2 : -INFINITY);   // exp2(-inf) = 0: no branch
  }
}

// Distortion sweeps: wave (pt, dir) accumulates M^T (values x its 16 probes)
// over the direction's children and sums (Z / Z_q(C)) D_q over its probes per
// child, scoring each child when the sweep reaches its cut.
template <typename T, int D, int QW>
__device__ void probe_sweeps(Ref<T, D>& U, const Dims& dm, const T* __restrict__ Kp, int n, int a, int b,
                             const int* XL, int nl, const int* XR, int nr, const uint32_t* qreg, int pt, float mq2,
                             float zc, float sc2) {
  using Lay = RefLds<T, D>;
  constexpr bool BF = Lay::BF;
  constexpr int DT = D / 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, i16 = lane & 15, g4 = lane >> 4;
  const bool prefix = wave < 4;
  const int nx = prefix ? nl : nr;
  if (16 * pt >= dm.W || nx == 0) return;
  const int q = 16 * pt + i16;
  const bool pok = q < dm.W;
  f32x4 M[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) M[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float Z = 0.f;
  float ev[4] = {0.f, 0.f, 0.f, 0.f};
  u32x2 eh = {0u, 0u}, em = {0u, 0u}, el = {0u, 0u};   // bf16 parts of the block's e
  u32x2 vop[BF ? DT : 1];                             // V^T operands of the block (bf16)
  float4 vf[BF ? 1 : DT];                             // ... (fp32)
  uint32_t kpre[QW];                                  // key quarter rows of the next block of the sweep
  int eblk = -1;
  const int lastblk = (n - 1) >> 4;
  block_k<T, D, QW>(Kp, n, prefix ? (a >> 4) : ((b - 1) >> 4), kpre);   // the sweep's first block
  int cur = prefix ? a : b;
  const float izc = 1.0f / zc;
  // scores child gc (prefix or suffix) from M and Z: (Z / Z_q(C)) D_q summed over
  // the wave's probes; z and v~ of the child were loaded before the sweep reached it
  auto score_child = [&](int gc, float z, const float4* vt) {
    const float Zs = col_sum4(Z);
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const float vv[4] = {vt[dt].x, vt[dt].y, vt[dt].z, vt[dt].w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float Mv = M[dt][r];
        const float df = Mv - z * vv[r];
        s1 += df * df;
        s2 += Mv * Mv;
      }
    }
    s1 = col_sum4(s1);
    s2 = col_sum4(s2);
    const float dz = Zs - z;
    const float Dq = dm.lam_Z * dz * dz * __builtin_amdgcn_rcpf(Zs * Zs + dm.eps) +
                     dm.lam_M * s1 * __builtin_amdgcn_rcpf(s2 + dm.eps);
    // sum over the wave's 16 probes (row 0 of the wave)
    const float con = row_sum16((g4 == 0 && pok) ? (Zs * izc) * Dq : 0.f);
    if (lane == 0) U.Con[gc * 4 + pt] = con;
  };
  for (int k = 0; k < nx; ++k) {
    const int c = prefix ? k : nx - 1 - k;
    const int x = prefix ? XL[c] : XR[c];
    const int gc = prefix ? c : CM + c;
    // accumulate the pieces between cur and x (each within one 16-token block)
    while (prefix ? cur < x : cur > x) {
      const int blk = prefix ? (cur >> 4) : ((cur - 1) >> 4);
      const int lo = prefix ? cur : max(x, blk << 4);
      const int hi = prefix ? min(x, (blk + 1) << 4) : cur;
      if (blk != eblk) {
        // sweeps visit consecutive blocks: this one was prefetched, the next one
        // goes in flight now (straight-line, so only the older loads are waited for)
        uint32_t kreg[QW];
#pragma unroll
        for (int h = 0; h < QW; ++h) kreg[h] = kpre[h];
        int nb = prefix ? blk + 1 : blk - 1;
        nb = nb < 0 ? 0 : (nb > lastblk ? lastblk : nb);
        block_k<T, D, QW>(Kp, n, nb, kpre);
        block_e<T, D, QW>(kreg, n, blk, qreg, mq2, pok, sc2, ev);
        if constexpr (BF) {
          split3x4(ev, eh, em, el);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const uint2 vv = *(const uint2*)(U.Vt + (16 * dt + i16) * Lay::LDV + 16 * blk + 4 * g4);
            vop[dt].x = vv.x;
            vop[dt].y = vv.y;
          }
        } else {
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            vf[dt] = *(const float4*)(U.Vt + (16 * dt + i16) * Lay::LDV + 16 * blk + 4 * g4);
        }
        eblk = blk;
      }
      const int t0 = 16 * blk + 4 * g4;
      bool in[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        in[r] = t0 + r >= lo && t0 + r < hi;
        Z += in[r] ? ev[r] : 0.f;
      }
      if constexpr (BF) {
        u32x2 mk;
        mk.x = (in[0] ? 0xffffu : 0u) | (in[1] ? 0xffff0000u : 0u);
        mk.y = (in[2] ? 0xffffu : 0u) | (in[3] ? 0xffff0000u : 0u);
        const s16x4 ph = as_op(eh & mk), pm = as_op(em & mk), pl = as_op(el & mk);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const s16x4 va = as_op(vop[dt]);
          M[dt] = mfma_bf16_16x16x16(va, pl, M[dt]);
          M[dt] = mfma_bf16_16x16x16(va, pm, M[dt]);
          M[dt] = mfma_bf16_16x16x16(va, ph, M[dt]);
        }
      } else {
        float emk[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) emk[r] = in[r] ? ev[r] : 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          M[dt] = mfma_f32_16x16x4(vf[dt].x, emk[0], M[dt]);
          M[dt] = mfma_f32_16x16x4(vf[dt].y, emk[1], M[dt]);
          M[dt] = mfma_f32_16x16x4(vf[dt].z, emk[2], M[dt]);
          M[dt] = mfma_f32_16x16x4(vf[dt].w, emk[3], M[dt]);
        }
      }
      if (prefix) cur = hi; else cur = lo;
    }
    if ((int)U.crow(0)[gc] >= 2) {
      const float zk = pok ? U.Zt[gc * WMAX + q] : 0.f;
      float4 vk[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vk[dt] = *(const float4*)(U.Vv + gc * D + 4 * g4 + 16 * dt);
      score_child(gc, zk, vk);
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(BT) void k_refine(const Dims* __restrict__ dmp, int mode, const T* __restrict__ K,
                                                const T* __restrict__ V, const T* __restrict__ Q,
                                                const float* __restrict__ cosT, const float* __restrict__ sinT,
                                                const int32_t* __restrict__ slot_starts,
                                                const int32_t* __restrict__ n_slots, const float* __restrict__ kappa,
                                                const TreeView* __restrict__ tvp) {
  // the argument structures are read from device memory where used (held in
  // scalar registers they would not fit)
  const Dims& dm = *dmp;
  const TreeView& tv = *tvp;
  using Lay = RefLds<T, D>;
  constexpr bool BF = Lay::BF;
  constexpr int H2 = D / 2;
  constexpr int QE = D / 4;
  constexpr int QW = BF ? QE / 2 : QE;
  extern __shared__ __align__(16) char smem[];
  Ref<T, D> U(smem);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, i16 = lane & 15, g4 = lane >> 4;
  const int J = *n_slots;
  const int nwork = tv.wctr[0];
  const uint64_t theta = mode == BUILD_FULL ? 0ull : tv.theta[0];
  const uint64_t theta_skip = mode == BUILD_FULL ? 0ull : tv.theta[1];
  const float scale = 1.0f / sqrtf((float)D);
  const int pt = wave & 3;                    // probe tile of this wave
  int* XL = U.xi;              // [0..31]  prefix cut list
  int* XR = U.xi + 32;         // [32..63] suffix cut list
  int* XB = U.xi + 64;         // [64..95] binary cuts
  int* meta = U.xi + 96;       // nXL, nXR, nXB, p, kmin bits, kmax bits, index of p in XL, of p+1 in XR,
                               // forced extraction (singleton floor)
  int* posL = U.xi + 128;      // index of XB[k] in XL
  int* posR = U.xi + 160;      // index of XB[k] in XR
  int* cnt = U.xi + 192;       // node count
  int* sw = U.xi + 193;        // current work item

  for (;;) {
    __syncthreads();
    if (tid == 0) sw[0] = atomicAdd(&tv.wctr[1], 1);
    __syncthreads();
    const int wi = sw[0];
    if (wi >= nwork) break;
    const int64_t unit = tv.work[8 * (int64_t)wi];
    const int lg = (int)(unit / dm.J_cap), j = (int)(unit % dm.J_cap);
    if (j >= J) continue;
    const int l = lg / dm.G, g = lg % dm.G;
    const int64_t a0 = slot_starts[j];
    const int n = slot_starts[j + 1] - (int)a0;
    if (n < 2 || n > NMAX || a0 < 0 || a0 + n > dm.N_c) continue;
    const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * a0;
    const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
    const T* Kp = K + ((int64_t)lg * dm.T + a0) * D;
    const T* Vp = V + ((int64_t)lg * dm.T + a0) * D;
    const T* Qp = Q + ((int64_t)l * dm.H + (int64_t)g * dm.hpg) * dm.W * D;
    const float w = tv.omega[lg];

    // the root's Split cannot be selected (its key bound is below the skip bound)
    const bool rskip = mode != BUILD_FULL &&
                       root_split_key_bound(w, tv.node_R[base], tv.node_D[base], ord) < theta_skip;
    // ---- node table; refine only nodes whose creating op reaches theta ----
    {
      const int nn0 = tv.unit_nn[unit];
      const uint64_t Eadd = tv.add_E[unit];
      bool any = false;
      for (int i = tid; i < nn0; i += BT) {
        const int64_t sl = base + i;
        U.na[i] = tv.node_a[sl] - (int)a0; U.nn[i] = tv.node_n[sl]; U.nc[i] = tv.node_child[sl];
        U.np[i] = tv.node_parent[sl]; U.nch[i] = tv.node_nch[sl]; U.nk[i] = tv.node_kind[sl];
        U.ncut[i] = tv.node_cut[sl]; U.nD[i] = tv.node_D[sl]; U.nR[i] = tv.node_R[sl]; U.nU[i] = tv.sp_U[sl];
        const uint64_t ec = U.np[i] < 0 ? Eadd : tv.sp_E[base + U.np[i]];
        U.nE[i] = ec;
        any |= U.nch[i] == 0 && U.nn[i] >= 2 && ec >= theta && (mode != BUILD_ROOT_SPLIT || i == 0) &&
               !(i == 0 && rskip);
      }
      if (tid == 0) cnt[0] = nn0;
      if (!__syncthreads_or(any)) continue;
    }

    // probe quarter rows of the wave's tile (probe q: window query q of head q mod |H(g)|)
    uint32_t qreg[QW];
    {
      const int q = 16 * pt + i16;
      const int uq = q < dm.W ? q : 0;
      const uint4* q4 = (const uint4*)(Qp + ((int64_t)(uq % dm.hpg) * dm.W + uq) * D + QE * g4);
#pragma unroll
      for (int h = 0; h < QW / 4; ++h) {
        const uint4 v = q4[h];
        qreg[4 * h] = v.x; qreg[4 * h + 1] = v.y; qreg[4 * h + 2] = v.z; qreg[4 * h + 3] = v.w;
      }
    }
    // ---- staging ----
    {
      // k° = RoPE^{-1}(k): item (token, 8-dim chunk of the first half) also
      // produces the partner dims d + D/2
      constexpr int CH = H2 / 8;
      for (int e = tid; e < n * CH; e += BT) {
        const int t = e / CH, c = 8 * (e % CH);
        const int64_t ta = a0 + t;
        const float4 c0 = *(const float4*)(cosT + ta * H2 + c), c1 = *(const float4*)(cosT + ta * H2 + c + 4);
        const float4 s0 = *(const float4*)(sinT + ta * H2 + c), s1 = *(const float4*)(sinT + ta * H2 + c + 4);
        float k1[8], k2[8];
        if constexpr (BF) {
          const uint4 u1 = *(const uint4*)(Kp + (int64_t)t * D + c);
          const uint4 u2 = *(const uint4*)(Kp + (int64_t)t * D + c + H2);
          const uint32_t w1[4] = {u1.x, u1.y, u1.z, u1.w}, w2[4] = {u2.x, u2.y, u2.z, u2.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            k1[2 * h] = __uint_as_float(w1[h] << 16); k1[2 * h + 1] = __uint_as_float(w1[h] & 0xffff0000u);
            k2[2 * h] = __uint_as_float(w2[h] << 16); k2[2 * h + 1] = __uint_as_float(w2[h] & 0xffff0000u);
          }
        } else {
          const float4* p1 = (const float4*)((const float*)Kp + (int64_t)t * D + c);
          const float4* p2 = (const float4*)((const float*)Kp + (int64_t)t * D + c + H2);
          const float4 a = p1[0], bq = p1[1], cq = p2[0], dq = p2[1];
          k1[0] = a.x; k1[1] = a.y; k1[2] = a.z; k1[3] = a.w; k1[4] = bq.x; k1[5] = bq.y; k1[6] = bq.z; k1[7] = bq.w;
          k2[0] = cq.x; k2[1] = cq.y; k2[2] = cq.z; k2[3] = cq.w; k2[4] = dq.x; k2[5] = dq.y; k2[6] = dq.z; k2[7] = dq.w;
        }
        const float cs8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
        const float sn8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        float o1[8], o2[8];
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          o1[h] = k1[h] * cs8[h] + k2[h] * sn8[h];
          o2[h] = k2[h] * cs8[h] - k1[h] * sn8[h];
        }
        float4* d1 = (float4*)(U.Ko + t * D + c);
        float4* d2 = (float4*)(U.Ko + t * D + c + H2);
        d1[0] = make_float4(o1[0], o1[1], o1[2], o1[3]); d1[1] = make_float4(o1[4], o1[5], o1[6], o1[7]);
        d2[0] = make_float4(o2[0], o2[1], o2[2], o2[3]); d2[1] = make_float4(o2[4], o2[5], o2[6], o2[7]);
        // ||k°_t||^2: the CH items of token t sit in CH consecutive lanes
        float ss = 0.f;
#pragma unroll
        for (int h = 0; h < 8; ++h) ss += o1[h] * o1[h] + o2[h] * o2[h];
#pragma unroll
        for (int o = 1; o < CH; o <<= 1) ss += __shfl_xor(ss, o, 64);
        if (e % CH == 0) U.Kn[t] = sqrtf(ss);
      }
      // V^T, zero past n
      const int rows16 = (n + 15) & ~15;
      if constexpr (BF) {
        constexpr int CPR = D / 8;
        for (int e = tid; e < (rows16 / 2) * CPR; e += BT) {
          const int grp = e / (8 * CPR), rem = e % (8 * CPR);
          const int c = rem / 8, t = 2 * (8 * grp + rem % 8);
          uint4 v0 = make_uint4(0, 0, 0, 0), v1 = v0;
          if (t < n) v0 = *(const uint4*)(Vp + (int64_t)t * D + 8 * c);
          if (t + 1 < n) v1 = *(const uint4*)(Vp + (int64_t)(t + 1) * D + 8 * c);
          const uint32_t pa[4] = {v0.x, v0.y, v0.z, v0.w}, pb[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            *(uint32_t*)(U.Vt + (8 * c + 2 * h) * Lay::LDV + t) = (pa[h] & 0xffffu) | (pb[h] << 16);
            *(uint32_t*)(U.Vt + (8 * c + 2 * h + 1) * Lay::LDV + t) = (pa[h] >> 16) | (pb[h] & 0xffff0000u);
          }
        }
      } else {
        constexpr int CPR = D / 4;
        for (int e = tid; e < rows16 * CPR; e += BT) {
          const int grp = e / (16 * CPR), rem = e % (16 * CPR);
          const int c = rem / 16, t = 16 * grp + rem % 16;
          float4 vv = make_float4(0.f, 0.f, 0.f, 0.f);
          if (t < n) vv = *(const float4*)((const float*)Vp + (int64_t)t * D + 4 * c);
          U.Vt[(4 * c + 0) * Lay::LDV + t] = vv.x;
          U.Vt[(4 * c + 1) * Lay::LDV + t] = vv.y;
          U.Vt[(4 * c + 2) * Lay::LDV + t] = vv.z;
          U.Vt[(4 * c + 3) * Lay::LDV + t] = vv.w;
        }
      }
      if (tid < n) {
        U.R[tid] = tv.tok_R[(int64_t)lg * dm.N_c + a0 + tid];
        U.A[tid] = tv.tok_A[(int64_t)lg * dm.N_c + a0 + tid];
        U.Kap[tid] = kappa[a0 + tid];
        U.fl[tid] = tv.fl_flag ? tv.fl_flag[(int64_t)lg * dm.N_c + a0 + tid] : 0;
      }
      if (tid < dm.W) {
        U.Mq[tid] = tv.probe_m[(int64_t)lg * dm.W + tid];
        U.Zc[tid] = tv.probe_ZC[(int64_t)lg * dm.W + tid];
      }
    }
    __syncthreads();
    float mq = 0.f, zc = 1.f;
    if (16 * pt + i16 < dm.W) { mq = U.Mq[16 * pt + i16]; zc = U.Zc[16 * pt + i16]; }
    // ---- top-down refinement in BFS order ----
    for (int head = 0;; ++head) {
      sync_after_lds_stores();               // the node table and cnt were stored at the end of the last pass
      const int count = cnt[0];
      if (head >= count || (mode == BUILD_ROOT_SPLIT && head > 0)) break;
      const int a = U.na[head], nv = U.nn[head], b = a + nv;
      if (nv < 2 || U.nch[head] > 0) continue;                  // leaf, or refined by an earlier pass
      if (mode != BUILD_FULL && (U.nE[head] < theta || (head == 0 && rskip))) continue;  // cannot reach the cut
      const float Dv = U.nD[head];
      if (nv == 2) {
        if (tid == 0) {
          const int c0 = count;
          U.nc[head] = c0; U.nch[head] = 2; U.nk[head] = 1; U.ncut[head] = (int)a0 + a + 1;
          for (int k = 0; k < 2; ++k) {
            U.na[c0 + k] = a + k; U.nn[c0 + k] = 1; U.nc[c0 + k] = -1; U.np[c0 + k] = head;
            U.nch[c0 + k] = 0; U.nk[c0 + k] = 0; U.ncut[c0 + k] = -1;
            U.nD[c0 + k] = 0.f; U.nR[c0 + k] = U.R[a + k];
          }
          cnt[0] = count + 2;
          if (mode != BUILD_FULL) {
            const float Us = utility(split_gain(w, U.nR[head], Dv, U.nD[c0] + U.nD[c0 + 1]), 1);
            const uint64_t k = op_key(Us, ord * 256u + 1u + (uint32_t)head);
            const uint64_t E = k < U.nE[head] ? k : U.nE[head];
            U.nU[head] = Us;
            U.nE[c0] = E; U.nE[c0 + 1] = E;
          }
        }
        continue;
      }
      // candidate flags over cut positions xi in (a, b)
      for (int t = tid; t < NMAX; t += BT) U.flag[t] = 0;
      __syncthreads();
      if (dm.k_curv > 0 && tid < nv - 1) {
        const int t = a + tid;                     // curvature position t -> cut t + 1
        const float kt = U.Kap[t];
        int rank = 0;
        // positions a .. b - 2, read eight at a time (all lanes read the same
        // words; the last read may run past b - 2 into the next LDS array, which
        // the position test masks), branch-free comparisons
        const int hi = b - 2;
        for (int t4 = a & ~3; t4 <= hi; t4 += 8) {
          const float4 k4 = *(const float4*)(U.Kap + t4);
          const float4 k5 = *(const float4*)(U.Kap + t4 + 4);
          const float kk[8] = {k4.x, k4.y, k4.z, k4.w, k5.x, k5.y, k5.z, k5.w};
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const int t2 = t4 + jj;
            rank += (int)((t2 >= a) & (t2 <= hi) & ((kk[jj] > kt) | ((kk[jj] == kt) & (t2 < t))));
          }
        }
        if (rank < dm.k_curv) U.flag[t + 1 - a] = 1;
      }
      if (tid == BT - 1) U.flag[nv / 2] = 1;      // midpoint a + floor(n/2)
      // curvature range and extraction token (wave 0)
      if (wave == 0) {
        float kmn = INFINITY, kmx = -INFINITY, best = -INFINITY, bestf = -INFINITY;
        int bi = 0x7fffffff, bf = 0x7fffffff;
        for (int t = a + lane; t < b; t += 64) {
          const float k = U.Kap[t];
          kmn = fminf(kmn, k);
          kmx = fmaxf(kmx, k);
          const float am = U.A[t];
          if (am > best || (am == best && t < bi)) { best = am; bi = t; }
          // singleton floor: the candidate of largest token value (App. A.3 split choice)
          if (U.fl[t] && (U.R[t] > bestf || (U.R[t] == bestf && t < bf))) { bestf = U.R[t]; bf = t; }
        }
        wave_minmax(kmn, kmx);
        wave_argmax(best, bi);
        wave_argmax(bestf, bf);
        if (lane == 0) {
          // a node of three or more tokens holding a floor candidate is extracted
          // there, with no choice
          const bool forced = bf != 0x7fffffff;
          meta[3] = forced ? bf : bi;
          meta[4] = __float_as_int(kmn);
          meta[5] = __float_as_int(kmx);
          meta[8] = forced ? 1 : 0;
        }
      }
      __syncthreads();
      // binary cuts XB (ascending) by ballot over the flags, then the prefix list
      // XL = XB + {p} (if p > a) and suffix list XR = XB + {p+1} (if p+1 < b)
      if (wave == 0) {
        const bool forced = meta[8] != 0;      // extraction only: no binary cut
        const bool f0 = !forced && lane >= 1 && lane < nv && U.flag[lane];
        const bool f1 = !forced && 64 + lane < nv && U.flag[64 + lane];
        const uint64_t m0 = __ballot(f0), m1 = __ballot(f1);
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        const int n0 = __popcll(m0);
        if (f0) XB[__popcll(m0 & below)] = a + lane;
        if (f1) XB[n0 + __popcll(m1 & below)] = a + 64 + lane;
        if (lane == 0) meta[2] = n0 + __popcll(m1);
      }
      __syncthreads();
      if (wave == 0) {
        const int nb = meta[2], p = meta[3];
        const bool on = lane < nb;
        const int xk = on ? XB[lane] : 0x7fffffff;
        const bool useP = p > a, useQ = p + 1 < b;
        const uint64_t lessP = __ballot(on && xk < p), eqP = __ballot(on && xk == p);
        const uint64_t lessQ = __ballot(on && xk < p + 1), eqQ = __ballot(on && xk == p + 1);
        const bool insL = useP && eqP == 0ull, insR = useQ && eqQ == 0ull;
        if (on) {
          const int pl = lane + ((insL && xk > p) ? 1 : 0);
          const int pr = lane + ((insR && xk > p + 1) ? 1 : 0);
          XL[pl] = xk; posL[lane] = pl;
          XR[pr] = xk; posR[lane] = pr;
        }
        if (lane == 0) {
          const int cp = __popcll(lessP), cq = __popcll(lessQ);
          if (insL) XL[cp] = p;
          if (insR) XR[cq] = p + 1;
          meta[0] = nb + (insL ? 1 : 0);
          meta[1] = nb + (insR ? 1 : 0);
          meta[6] = useP ? cp : -1;         // index of p in XL ([a, p))
          meta[7] = useQ ? cq : -1;         // index of p + 1 in XR ([p+1, b))
        }
      }
      __syncthreads();
      const int nl = meta[0], nr = meta[1], nb = meta[2], p = meta[3];
      proto_sums<T, D>(U, dm, a, b, XL, nl, XR, nr);
      __syncthreads();
      proto_keys<T, D>(U, dm, a0, a, b, XL, nl, XR, nr, cosT, sinT);
      __syncthreads();
      proto_attention<T, D, QW>(U, dm, nl, nr, qreg, pt, scale);
      __syncthreads();
      probe_sweeps<T, D, QW>(U, dm, Kp, n, a, b, XL, nl, XR, nr, qreg, pt, mq * 1.44269504088896341f, zc,
                             scale * 1.44269504088896341f);
      __syncthreads();
      // D of each child: mean over probes (fixed order)
      if (tid < nl + nr) {
        const int gc = tid < nl ? tid : CM + (tid - nl);
        float acc = 0.f;
        if ((int)U.crow(0)[gc] >= 2) {
          for (int p4 = 0; p4 < 4 && 16 * p4 < dm.W; ++p4) acc += U.Con[gc * 4 + p4];
          acc /= (float)dm.W;
        }
        U.crow(4)[gc] = acc;
      }
      __syncthreads();
      // scores (fp32): best binary cut by a wave-0 argmax (smaller cut wins ties),
      // then the extraction score and the append by lane 0
      if (wave == 0) {
        const float* cD = U.crow(4);
        const float* cRr = U.crow(1);
        const float kmn = __int_as_float(meta[4]), kmx = __int_as_float(meta[5]);
        const float kr = kmx - kmn;
        float best = -INFINITY;
        int bk = 0x7fffffff;
        if (lane < nb) {
          const int x = XB[lane];
          const float kh = kr > 0.f ? (U.Kap[x - 1] - kmn) / kr : 0.f;
          best = ((Dv - cD[posL[lane]]) - cD[CM + posR[lane]]) + dm.lam_kappa * kh;
          bk = lane;
        }
        wave_argmax(best, bk);
        if (lane == 0) {
          const int iL = meta[6], iR = meta[7];
          float dsum = 0.f;
          int nkid = 1;
          if (p > a) { dsum += cD[iL]; ++nkid; }
          if (p + 1 < b) { dsum += cD[CM + iR]; ++nkid; }
          const float gext = (Dv - dsum) / (float)(nkid - 1);
          const int c0 = count;
          U.nc[head] = c0;
          int c = c0;
          if (best >= gext) {
            const int bx = XB[bk];
            U.nch[head] = 2; U.nk[head] = 1; U.ncut[head] = (int)a0 + bx;
            U.na[c] = a; U.nn[c] = bx - a; U.nD[c] = cD[posL[bk]]; U.nR[c] = cRr[posL[bk]]; ++c;
            U.na[c] = bx; U.nn[c] = b - bx; U.nD[c] = cD[CM + posR[bk]]; U.nR[c] = cRr[CM + posR[bk]]; ++c;
          } else {
            U.nch[head] = (uint8_t)nkid; U.nk[head] = 2; U.ncut[head] = (int)a0 + p;
            if (p > a) { U.na[c] = a; U.nn[c] = p - a; U.nD[c] = cD[iL]; U.nR[c] = cRr[iL]; ++c; }
            U.na[c] = p; U.nn[c] = 1; U.nD[c] = 0.f; U.nR[c] = U.R[p]; ++c;
            if (p + 1 < b) { U.na[c] = p + 1; U.nn[c] = b - p - 1; U.nD[c] = cD[CM + iR]; U.nR[c] = cRr[CM + iR]; ++c; }
          }
          for (int k = c0; k < c; ++k) { U.nc[k] = -1; U.np[k] = head; U.nch[k] = 0; U.nk[k] = 0; U.ncut[k] = -1; }
          cnt[0] = c;
          if (mode != BUILD_FULL) {
            float sd = 0.f;
            for (int k = c0; k < c; ++k) sd += U.nD[k];
            const float Us = utility(split_gain(w, U.nR[head], Dv, sd), c - c0 - 1);
            const uint64_t kk = op_key(Us, ord * 256u + 1u + (uint32_t)head);
            const uint64_t E = kk < U.nE[head] ? kk : U.nE[head];
            U.nU[head] = Us;
            for (int k = c0; k < c; ++k) U.nE[k] = E;
          }
        }
      }
    }
    __syncthreads();
    // ---- write the node table ----
    const int count = cnt[0];
    for (int i = tid; i < 2 * n; i += BT) {
      const int64_t sl = base + i;
      if (i < count) {
        tv.node_a[sl] = (int32_t)a0 + U.na[i];
        tv.node_n[sl] = U.nn[i];
        tv.node_child[sl] = U.nc[i];
        tv.node_parent[sl] = U.np[i];
        tv.node_nch[sl] = U.nch[i];
        tv.node_kind[sl] = U.nk[i];
        tv.node_cut[sl] = U.ncut[i];
        tv.node_D[sl] = U.nD[i];
        tv.node_R[sl] = U.nR[i];
        if (mode != BUILD_FULL) {          // keys of the Splits known so far (refined nodes)
          const int c = U.nch[i];
          if (c > 0) {
            const uint64_t k = op_key(U.nU[i], ord * 256u + 1u + (uint32_t)i);
            tv.sp_U[sl] = U.nU[i];
            tv.sp_E[sl] = k < U.nE[i] ? k : U.nE[i];
            tv.sp_cost[sl] = (uint8_t)(c - 1);
          } else {
            tv.sp_U[sl] = 0.f;
            tv.sp_E[sl] = 0;
            tv.sp_cost[sl] = 0;
          }
          tv.sp_exec[sl] = 0;
        }
      } else {
        tv.sp_cost[sl] = 0;
        tv.sp_E[sl] = 0;
        tv.sp_exec[sl] = 0;
      }
    }
    if (tid == 0) tv.unit_nn[unit] = count;
  }
}

// ---- work list: the units with a node to refine ---------------------------
__global__ void k_work_reset(TreeView tv) {
  if (threadIdx.x < 4) tv.wctr[threadIdx.x] = 0;
}

// Lists the units to refine whose slot length lies in [n_lo, n_hi): the
// launches go from long slots to short ones, so the persistent workgroups take
// the long (slow) items first and finish together.
__global__ void k_work_mark(Dims dm, int mode, TreeView tv, int n_lo, int n_hi) {
  const int64_t unit = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (unit >= (int64_t)dm.L * dm.G * dm.J_cap) return;
  const int lg = (int)(unit / dm.J_cap), j = (int)(unit % dm.J_cap);
  const int J = *tv.nslots;
  if (j >= J || J > dm.J_cap) return;
  const int64_t a0 = tv.slots[j];
  const int ns = tv.slots[j + 1] - (int)a0;
  if (ns < n_lo || ns >= n_hi) return;
  const int64_t base = (int64_t)lg * 2 * dm.N_c + 2 * a0;
  const int nn = tv.unit_nn[unit];
  const uint64_t theta = (mode == BUILD_FULL || mode == BUILD_ROOT_FULL) ? 0ull : tv.theta[0];
  bool need = false;
  for (int i = 0; i < nn && !need; ++i) {
    if ((mode == BUILD_ROOT_SPLIT || mode == BUILD_ROOT_FULL) && i > 0) break;
    const int64_t s = base + i;
    if (tv.node_nch[s] != 0 || tv.node_n[s] < 2) continue;
    if (mode == BUILD_FULL || mode == BUILD_ROOT_FULL) { need = true; break; }
    const int par = tv.node_parent[s];
    if (par < 0) {                          // the root: its Add reaches theta and its Split may
      const uint32_t ord = (uint32_t)lg * (uint32_t)J + (uint32_t)j;
      need = tv.add_E[unit] >= theta &&
             root_split_key_bound(tv.omega[lg], tv.node_R[s], tv.node_D[s], ord) >= tv.theta[1];
    } else {
      need = tv.sp_E[base + par] >= theta;
    }
  }
  if (need) {
    // the item carries what the refinement of the root reads first, so a
    // workgroup needs one load instead of a chain of dependent ones
    const int pos = atomicAdd(&tv.wctr[0], 1);
    const uint64_t Ea = tv.add_E[unit];
    int4* it = (int4*)(tv.work + 8 * (int64_t)pos);
    it[0] = make_int4((int32_t)unit, (int32_t)a0, tv.node_n[base], __float_as_int(tv.node_D[base]));
    it[1] = make_int4(__float_as_int(tv.node_R[base]), __float_as_int(tv.omega[lg]), (int32_t)(uint32_t)Ea,
                      (int32_t)(uint32_t)(Ea >> 32));
  }
}

static int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cus[dev] = v;
  }
  return cus[dev];
}

hipError_t launch_build(const Dims& dm, int lds_bytes, int mode, const void* K, const void* V, const void* Q,
                        const float* cosT, const float* sinT, const int32_t* slot_starts, const int32_t* n_slots,
                        const float* kappa, const TreeView& tv, hipStream_t st, bool listed) {
  if (!listed) {                            // else the level passes left the work list
    const int64_t units = (int64_t)dm.L * dm.G * dm.J_cap;
    hipLaunchKernelGGL(k_work_reset, dim3(1), dim3(64), 0, st, tv);
    const unsigned mb = (unsigned)((units + 255) / 256);
    hipLaunchKernelGGL(k_work_mark, dim3(mb), dim3(256), 0, st, dm, mode, tv, 96, NMAX + 1);
    hipLaunchKernelGGL(k_work_mark, dim3(mb), dim3(256), 0, st, dm, mode, tv, 48, 96);
    hipLaunchKernelGGL(k_work_mark, dim3(mb), dim3(256), 0, st, dm, mode, tv, 0, 48);
  }
  const bool roots = mode == BUILD_ROOT_SPLIT || mode == BUILD_ROOT_FULL;
  if (dm.dtype == GRACEKV_BF16 && roots)
    return launch_split_root(dm, mode, K, V, Q, cosT, sinT, slot_starts, n_slots, kappa, tv, 2 * device_cus(), st);
  const dim3 grid((unsigned)device_cus());
#define GKV_LAUNCH_REFINE(TT, DD)                                                                          \
  do {                                                                                                     \
    auto fn = k_refine<TT, DD>;                                                                            \
    hipError_t e0 = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes); \
    if (e0 != hipSuccess) return e0;                                                                       \
    hipLaunchKernelGGL(fn, grid, dim3(BT), lds_bytes, st, (const Dims*)tv.kargs, mode, (const TT*)K,         \
                       (const TT*)V, (const TT*)Q, cosT, sinT, slot_starts, n_slots, kappa,                \
                       (const TreeView*)((const char*)tv.kargs + 512));                                    \
  } while (0)
  if (dm.dtype == GRACEKV_BF16) {
    if (dm.d == 128) GKV_LAUNCH_REFINE(uint16_t, 128); else GKV_LAUNCH_REFINE(uint16_t, 64);
  } else {
    if (dm.d == 128) GKV_LAUNCH_REFINE(float, 128); else GKV_LAUNCH_REFINE(float, 64);
  }
#undef GKV_LAUNCH_REFINE
  return hipGetLastError();
}

hipError_t launch_levels_bf16(const Dims& dm, bool full, const void* K, const void* V, const void* Q,
                              const float* cosT, const float* sinT, const int32_t* slot_starts,
                              const int32_t* n_slots, const float* kappa, const TreeView& tv, hipStream_t st) {
  return launch_levels(dm, full, K, V, Q, cosT, sinT, slot_starts, n_slots, kappa, tv, 2 * device_cus(), st);
}

}  // namespace gkv
