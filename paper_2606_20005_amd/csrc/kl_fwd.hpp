// Forward kernels of the fused attention-KL (Algorithm 1, Sec. 3.2).
//
// A wave keeps 32 query rows of Q_a and Q_b in registers as MFMA B operands
// and walks the key tiles K_a, K_b (32 rows each) that its workgroup streams
// through an LDS ring. Per tile it forms S_a^T = K_a Q_a^T and S_b^T =
// K_b Q_b^T on the 32x32x16 bf16 MFMA with fp32 accumulation. In the
// transposed result a lane owns one query row (column l % 32) and 16 keys of
// the tile, so every row reduction is in-lane: the two half-waves (l / 32 =
// 0, 1) hold disjoint key subsets of the same rows and each keeps its own five
// running scalars, merged once at the end by the split-K rule of Sec. 3.3.
// Nothing crosses lanes inside the key loop. Every kFoldTiles tiles a lane
// also folds its scalars into a per-lane total in LDS by the same rule, which
// bounds the number of additions any fp32 running sum takes.
//
// Arithmetic is in the base-2 domain (Sec. 5 uses exp2): t = raw * s * log2(e),
// p = 2^(t - u) for an exponent reference u, and acc = sum p_a (t_a - t_b)
// (eq:acc-invariant in base 2, so acc * ln 2 is the paper's acc). Per
// element: one fma and one exp2 per distribution, two adds and a sub + fma
// for acc. The tile maxima and the rescaling of Algorithm 1 run only when a
// row's reference has to move (the lazy reference, below).
//
// Masking. Causal key tiles past a row block's frontier are never loaded.
// On tiles that cross the diagonal or the ragged key tail, the raw logits of
// keys a row may not see are replaced by kMaskedRaw, a finite stand-in for
// -inf: such a key gets p = 2^(c * kMaskedRaw - u) = 0 exactly and a finite
// log-ratio, so p * (x_a - x_b) = 0 and the update needs no per-key test.
// In the exact update a half-wave whose keys so far were all masked has a
// maximum below kNoKeyRaw and takes 0 as its exponent reference. This needs
// |raw logits| < 1e29 and s * log2(e) * 1e30 finite, far beyond any bf16
// attention input.
//
// "a" is the distribution in the first KL slot, "b" the second: the host
// passes (Q1,K1) as a for KL(P1||P2) and swaps the roles for KL(P2||P1).
//
// One kernel serves every head-dim pair; its configuration (waves per
// workgroup, workgroups per CU, key-tile layout) is chosen per pair at the
// end of this file. Every wave forms its own logits and runs its own online update:
// on gfx950 this update is bound by vector and transcendental issue (two
// exp2 per pair), and variants that hand the matrix work to separate waves
// in barrier-separated phases measured slower (an MFMA stream slows the
// vector waves of its SIMD by about a quarter, and a single wave issues its
// vector instructions at a fraction of the SIMD's rate).
#pragma once

#include <type_traits>

#include "kl_common.hpp"

namespace streamkl {

constexpr int kFwdBK = 32;             // key rows per tile (one 32x32 MFMA block)
constexpr float kMaskedRaw = -1e30f;   // raw logit of a key the row may not see
constexpr float kNoKeyRaw = -5e29f;    // maxima below this mean "no visible key yet"

// Five running row scalars of one half-wave. mra, mrb: the raw maximum at
// the last exact update (s > 0, so the scaled one is c * m), -inf while the
// half-wave has seen no visible key; it sets the exponent reference u = c m,
// and l and acc are relative to 2^u (base-2 domain, see above).
struct RowState {
  float mra, la, mrb, lb, acc;
};

// Per-tile values of the update: the negated exponent references and the
// tile's partial sums (two interleaved chains each).
struct TileCarry {
  float ua, ub;   // negated exponent references of this tile
  float la[2], lb[2], ac[2];
};

// Replace the raw logits of keys outside [0, klimit_excl) or past
// kcausal_max by kMaskedRaw. Register i of the transposed MFMA result holds
// key kbase + 8 (i / 4) + i % 4, kbase = first key of the tile + 4 * half.
__device__ __forceinline__ void mask_tile(f32x16& sa, f32x16& sb, int kbase, int klimit_excl, int kcausal_max) {
  const int kmax = min(klimit_excl - 1, kcausal_max);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const bool ok = kbase + 8 * (i >> 2) + (i & 3) <= kmax;
    sa[i] = ok ? sa[i] : kMaskedRaw;
    sb[i] = ok ? sb[i] : kMaskedRaw;
  }
}

__device__ __forceinline__ void fwd_element(TileCarry& tc, float ra, float rb, float ca, float cb, int slot,
                                            bool first) {
  const float xa = __builtin_fmaf(ra, ca, tc.ua);
  const float xb = __builtin_fmaf(rb, cb, tc.ub);
  const float pa = exp2_fast(xa);
  const float pb = exp2_fast(xb);
  const float d = xa - xb;
  if (first) {
    tc.la[slot] = pa;
    tc.lb[slot] = pb;
    tc.ac[slot] = pa * d;
  } else {
    tc.la[slot] += pa;
    tc.lb[slot] += pb;
    tc.ac[slot] = __builtin_fmaf(pa, d, tc.ac[slot]);
  }
}

// Lazy exponent reference. The running sums of a row stay exact for any
// exponent reference that is actually applied, as long as every term
// 2^(x - u) and every sum stays in the fp32 range: the reference need not be
// the running maximum. So each tile is first reduced against the references
// the state already holds (u = c m, m the raw maximum at the last exact
// update), without its maxima and without rescaling. A masked key still gives
// 0: its stand-in logit lies about 1e30 below any real reference. A lane
// keeps that result only if its two tile sums add up to at most kLazySumMax,
// which also rules out inf and NaN, and a half-wave with no reference yet
// (m = -inf) always overflows. A wave with a lane that fails forms the tile's logits
// again from the stage and runs the exact update on the failing lanes alone:
// the first tile of every pass, and a tile whose keys rise more than about 64
// doublings above the reference. A row's result depends on its own data only.
constexpr float kLazySumMax = 0x1p64f;

// Online update of one tile (Algorithm 1). exact (wave-uniform): form the new
// row maxima over the lane's 16 keys and rescale the sums to them first;
// otherwise reduce against the held references. Returns whether the lane
// took the tile. tc.ua, tc.ub hold the negated references -u.
__device__ __forceinline__ bool fwd_update(RowState& st, TileCarry& tc, const f32x16& sa, const f32x16& sb,
                                           float ca, float cb, bool exact) {
  if (exact) {
    float xa = st.mra, xb = st.mrb;
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      xa = fmaxf(fmaxf(xa, sa[i]), sa[i + 1]);
      xb = fmaxf(fmaxf(xb, sb[i]), sb[i + 1]);
    }
    tc.ua = xa < kNoKeyRaw ? 0.f : -ca * xa;
    tc.ub = xb < kNoKeyRaw ? 0.f : -cb * xb;
    // 2^(m_old - m_new); 0 while m_old is -inf or a masked stand-in
    const float aa = exp2_fast(__builtin_fmaf(ca, st.mra, tc.ua));
    const float ab = exp2_fast(__builtin_fmaf(cb, st.mrb, tc.ub));
    // a half-wave with no visible key yet keeps -inf, so that a lazy pass on
    // it overflows and falls back to this update
    st.mra = xa < kNoKeyRaw ? kNegInf : xa;
    st.mrb = xb < kNoKeyRaw ? kNegInf : xb;
    st.la *= aa;
    st.lb *= ab;
    st.acc *= aa;
  } else {
    tc.ua = -ca * st.mra;
    tc.ub = -cb * st.mrb;
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) fwd_element(tc, sa[i], sb[i], ca, cb, i & 1, i < 2);
  const float tla = tc.la[0] + tc.la[1], tlb = tc.lb[0] + tc.lb[1];
  // both sums are >= 0: their sum bounds each, and an inf or NaN in either fails
  const bool ok = exact || tla + tlb <= kLazySumMax;
  // sum p_a (t_a - t_b) = sum p_a (x_a - x_b) + (u_a - u_b) sum p_a
  const float dacc = __builtin_fmaf(tc.ub - tc.ua, tla, tc.ac[0] + tc.ac[1]);
  st.la = ok ? st.la + tla : st.la;
  st.lb = ok ? st.lb + tlb : st.lb;
  st.acc = ok ? st.acc + dacc : st.acc;
  return ok;
}

// S^T of one key tile on the MFMA: A = key rows from LDS (the tile's rows of
// K_a from tile_a, of K_b from tile_b), B = the lane's resident query rows;
// the two accumulation chains alternate. PAD: the tile is in the row-padded
// layout and base_a, base_b are the lane's operand bases (chunk slots);
// otherwise it is swizzled and the addresses are recomputed here.
template <int DA, int DB, bool PAD, int LA = 4>
__device__ __forceinline__ void fwd_logits(const u32x4* tile_a, const u32x4* tile_b, const bf16x8 (&qa)[DA / 16],
                                           const bf16x8 (&qb)[DB / 16], f32x16& sa, f32x16& sb, int lane,
                                           int base_a, int base_b) {
  constexpr int KA = DA / 16, KB = DB / 16, KM = KA > KB ? KA : KB;
  constexpr int CA = DA / 8, CB = DB / 8;
  f32x16 acc_a = zero16(), acc_b = zero16();
  if constexpr (PAD) {
    const u32x4* ta = tile_a + base_a;
    const u32x4* tb = tile_b + base_b;
#pragma unroll
    for (int ks = 0; ks < KM; ++ks) {
      if (ks < KA) acc_a = mfma32(__builtin_bit_cast(bf16x8, ta[ks]), qa[ks], acc_a);
      if (ks < KB) acc_b = mfma32(__builtin_bit_cast(bf16x8, tb[ks]), qb[ks], acc_b);
    }
  } else {
    const int half = lane >> 5;
    // Recompute the swizzled operand addresses on every call rather than keep
    // them live across the loop: the update state has no registers to spare.
    int r = lane & 31;
    asm volatile("" : "+v"(r));
    const u32x4* ta = tile_a;
    const u32x4* tb = tile_b;
#pragma unroll
    for (int ks = 0; ks < KM; ++ks) {
      if (ks < KA) acc_a = mfma32(lds_row8<CA>(ta, r, 2 * ks + half), qa[ks], acc_a);
      if (ks < KB) acc_b = mfma32(lds_row8<CB>(tb, r, 2 * ks + half), qb[ks], acc_b);
    }
  }
  // Keep LOOKAHEAD (at most LA) operand reads in flight ahead of the MFMA
  // that consumes them: with one logits wave per SIMD nothing else hides the
  // LDS latency.
  constexpr int NM = KA + KB, LOOKAHEAD = NM < LA ? NM : LA;
  __builtin_amdgcn_sched_group_barrier(0x100, LOOKAHEAD, 0);   // LDS reads
#pragma unroll
  for (int i = 0; i < NM - LOOKAHEAD; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);         // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);         // one LDS read
  }
  __builtin_amdgcn_sched_group_barrier(0x008, LOOKAHEAD, 0);
  sa = acc_a;
  sb = acc_b;
}

// Q rows of this lane as MFMA B operands: chunk 2 * ks + half of row myq.
// dreal: the row length in global memory (D, or less for a padded head dim:
// the chunks past it are zeros).
template <int D>
__device__ __forceinline__ void load_q_operands(bf16x8 (&q)[D / 16], const uint16_t* Q, size_t bh, int NQ, int myq,
                                                int half, int dreal) {
  const bool okq = myq < NQ;
  const u32x4* p = reinterpret_cast<const u32x4*>(Q + (bh * NQ + (okq ? myq : 0)) * dreal);
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const int c = 2 * ks + half;
    q[ks] = __builtin_bit_cast(bf16x8, okq && 8 * c < dreal ? p[c] : u32x4{0u, 0u, 0u, 0u});
  }
}

// Five row statistics with the maxima scaled to the base-2 exponent domain
// (m = c * raw maximum, -inf when the row has seen no key): the partial state
// of Sec. 3.3, which merges associatively.
struct RowPartial {
  float ma, la, mb, lb, acc;
};

// Split-K merge (Sec. 3.3) of two partial states of the same row.
__device__ __forceinline__ RowPartial merge_partials(const RowPartial& x, const RowPartial& y) {
  RowPartial r;
  r.ma = fmaxf(x.ma, y.ma);
  r.mb = fmaxf(x.mb, y.mb);
  if (r.ma == kNegInf) return RowPartial{kNegInf, 0.f, kNegInf, 0.f, 0.f};
  const float fx = exp2_fast(x.ma - r.ma), fy = exp2_fast(y.ma - r.ma);
  const float gx = exp2_fast(x.mb - r.mb), gy = exp2_fast(y.mb - r.mb);
  r.la = x.la * fx + y.la * fy;
  r.lb = x.lb * gx + y.lb * gy;
  r.acc = x.acc * fx + y.acc * fy;
  return r;
}

// The running state of a half-wave as a partial state.
__device__ __forceinline__ RowPartial state_partial(const RowState& st, float ca, float cb) {
  auto scaled = [](float c, float m) { return m < kNoKeyRaw ? kNegInf : c * m; };
  return RowPartial{scaled(ca, st.mra), st.la, scaled(cb, st.mrb), st.lb, st.acc};
}

// Merge the partial states of the two half-waves of each row; lanes of both
// halves return the row's partial state.
__device__ __forceinline__ RowPartial halfwave_merge(const RowPartial& mine) {
  const RowPartial other{__shfl_xor(mine.ma, 32), __shfl_xor(mine.la, 32), __shfl_xor(mine.mb, 32),
                         __shfl_xor(mine.lb, 32), __shfl_xor(mine.acc, 32)};
  return merge_partials(mine, other);
}

// Key tiles per chunk of the running sums. Every kFoldTiles tiles a lane
// merges its running state into a per-lane total kept in LDS (the merge rule
// of Sec. 3.3) and restarts from the empty state, so no fp32 running sum
// takes more than kFoldTiles additions: adding ever smaller tile sums to one
// large fp32 total drifts systematically (about 1% on the KL of 4M-key rows,
// against 1e-6 for the chunked sums).
constexpr int kFoldTiles = 64;

// KL (eq:kl-final), LSE_a and LSE_b (natural log) of a row from its complete
// state: LSE_t = (m_t + log2 l_t) ln 2 and KL = acc ln 2 / l_a + LSE_b - LSE_a.
__device__ __forceinline__ void write_row(const RowPartial& p, size_t ri, float* __restrict__ kl,
                                          float* __restrict__ lse_a, float* __restrict__ lse_b) {
  float out_kl = 0.f, out_la = kNegInf, out_lb = kNegInf;
  if (p.ma != kNegInf) {
    out_la = (p.ma + log2f(p.la)) * kLn2;
    out_lb = (p.mb + log2f(p.lb)) * kLn2;
    out_kl = p.acc * kLn2 / p.la + out_lb - out_la;
  }
  kl[ri] = out_kl;
  lse_a[ri] = out_la;
  lse_b[ri] = out_lb;
}

// Per-row arithmetic of the online pass, as a policy of fwd_pass.
// SoftmaxRows keeps the five running scalars of Algorithm 1; SigmoidRows
// keeps the sums of the sigmoid-score divergence. Each provides: State
// (what a lane carries across tiles), Partial (what it stores, merges and
// returns), init, reset (start a chunk), update (one tile, lazy or exact;
// returns whether the lane took it), partial, merge, and the NTOT floats per
// thread that a chunk total takes in LDS.
struct SoftmaxRows {
  static constexpr int NTOT = 5;
  struct State {
    RowState st;
    TileCarry tc;
  };
  typedef RowPartial Partial;
  __device__ __forceinline__ static State init() { return State{RowState{kNegInf, 0.f, kNegInf, 0.f, 0.f}, {}}; }
  // a new chunk keeps the exponent references (any applied reference is exact)
  __device__ __forceinline__ static void reset(State& s) { s.st = RowState{s.st.mra, 0.f, s.st.mrb, 0.f, 0.f}; }
  // exact = false: the lazy update; returns whether this lane took the tile
  __device__ __forceinline__ static bool update(State& s, const f32x16& sa, const f32x16& sb, float ca, float cb,
                                                bool exact) {
    return fwd_update(s.st, s.tc, sa, sb, ca, cb, exact);
  }
  __device__ __forceinline__ static Partial partial(const State& s, float ca, float cb) {
    return state_partial(s.st, ca, cb);
  }
  __device__ __forceinline__ static Partial merge(const Partial& x, const Partial& y) { return merge_partials(x, y); }
  __device__ __forceinline__ static void store(float* tot, int i, int n, const Partial& r) {
    tot[i] = r.ma;
    tot[n + i] = r.la;
    tot[2 * n + i] = r.mb;
    tot[3 * n + i] = r.lb;
    tot[4 * n + i] = r.acc;
  }
  __device__ __forceinline__ static Partial load(const float* tot, int i, int n) {
    return Partial{tot[i], tot[n + i], tot[2 * n + i], tot[3 * n + i], tot[4 * n + i]};
  }
  __device__ __forceinline__ static Partial halfwave(const Partial& p) { return halfwave_merge(p); }
};

// Sigmoid scores (Sec. 3.1, "Generalizability beyond Softmax"): A_t =
// sigmoid(S_t) with no normalisation, and the row value is the generalized
// KL sum_j [A_a log(A_a / A_b) - A_a + A_b] over the visible keys. With
// lr = log2(A_a / A_b) (sigmoid_pair) a lane keeps four plain sums over its
// keys: acc = sum A_a lr (base 2), dif = sum (A_b - A_a) and the masses
// sum A_a, sum A_b; L = acc ln 2 + dif. No maximum or rescaling is needed:
// every term is bounded (A <= 1, |lr| <= |za| + |zb| + 1). Chunk totals and
// the two half-waves combine by addition.
struct SigmoidPartial {
  float acc, dif, ma, mb;
};

struct SigmoidRows {
  static constexpr int NTOT = 4;
  typedef SigmoidPartial State;
  typedef SigmoidPartial Partial;
  __device__ __forceinline__ static State init() { return State{0.f, 0.f, 0.f, 0.f}; }
  __device__ __forceinline__ static void reset(State& s) { s = init(); }
  // no reference to keep: every tile is taken
  __device__ __forceinline__ static bool update(State& s, const f32x16& sa, const f32x16& sb, float ca, float cb,
                                                bool) {
    float acc[2] = {0.f, 0.f}, dif[2] = {0.f, 0.f}, ma[2] = {0.f, 0.f}, mb[2] = {0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const SigmoidPair t = sigmoid_pair(sa[i] * ca, sb[i] * cb);
      const int k = i & 1;
      acc[k] = __builtin_fmaf(t.a, t.lr, acc[k]);
      dif[k] += t.b - t.a;
      ma[k] += t.a;
      mb[k] += t.b;
    }
    s.acc += acc[0] + acc[1];
    s.dif += dif[0] + dif[1];
    s.ma += ma[0] + ma[1];
    s.mb += mb[0] + mb[1];
    return true;
  }
  __device__ __forceinline__ static Partial partial(const State& s, float, float) { return s; }
  __device__ __forceinline__ static Partial merge(const Partial& x, const Partial& y) {
    return Partial{x.acc + y.acc, x.dif + y.dif, x.ma + y.ma, x.mb + y.mb};
  }
  __device__ __forceinline__ static void store(float* tot, int i, int n, const Partial& r) {
    tot[i] = r.acc;
    tot[n + i] = r.dif;
    tot[2 * n + i] = r.ma;
    tot[3 * n + i] = r.mb;
  }
  __device__ __forceinline__ static Partial load(const float* tot, int i, int n) {
    return Partial{tot[i], tot[n + i], tot[2 * n + i], tot[3 * n + i]};
  }
  __device__ __forceinline__ static Partial halfwave(const Partial& p) {
    return merge(p, Partial{__shfl_xor(p.acc, 32), __shfl_xor(p.dif, 32), __shfl_xor(p.ma, 32), __shfl_xor(p.mb, 32)});
  }
};

// L and the masses of a complete sigmoid row; the masses are written where
// the caller asked for them.
__device__ __forceinline__ void write_row_sigmoid(const SigmoidPartial& p, size_t ri, float* __restrict__ kl,
                                                  float* __restrict__ mass_a, float* __restrict__ mass_b) {
  kl[ri] = __builtin_fmaf(p.acc, kLn2, p.dif);
  if (mass_a) mass_a[ri] = p.ma;
  if (mass_b) mass_b[ri] = p.mb;
}

// Row geometry shared by both kernels. Tiles 0 .. tlast hold keys some row of
// the wave may see (-1: none); tiles from tmask on cross the causal diagonal
// of some row of the wave or the ragged key tail.
struct WaveTiles {
  int tlast, tmask;
};

template <bool CAUSAL>
__device__ __forceinline__ WaveTiles wave_tiles(int qw, int wlast, int NQ, int NK, int ntiles) {
  const int off = NK - NQ;
  int tlast = qw < NQ ? ntiles - 1 : -1;
  int tmask = NK / kFwdBK;
  if (CAUSAL) {
    // last tile holding a key of the wave's last row (none if even that row sees no key)
    tlast = wlast + off < 0 ? -1 : min(tlast, (wlast + off) / kFwdBK);
    // first tile whose last key lies past the frontier of the wave's first row
    tmask = qw + off + 1 <= 0 ? 0 : min(tmask, (qw + off + 1) / kFwdBK);
  }
  return WaveTiles{__builtin_amdgcn_readfirstlane(tlast), __builtin_amdgcn_readfirstlane(tmask)};
}

// ----------------------------------------------------------------------------
// Forward kernel. A workgroup of NW waves owns 32 * NW / KS query rows and
// streams the key tiles once for all of them (the first DMA_NT threads issue
// the loads). With KS = 1 each wave forms and reduces every tile for its 32
// rows. With KS = 2 a ring stage holds two consecutive tiles and the waves
// split in two halves over the same rows: wave w (row group w % RG) takes the
// first tile of each stage when w < RG, the second otherwise, and the two
// halves merge their row states once at the end by the split-K rule. Stage
// iteration u forms and reduces stage u while stage u + NSTAGE - 1 streams
// into the buffer stage u - 1 occupied.
// ----------------------------------------------------------------------------
template <int DA_, int DB_, int NSTAGE_, int MINB_, int NW_ = 4, bool PAD_ = false, int KS_ = 1>
struct FwdTraits {
  static constexpr int DA = DA_, DB = DB_;
  static constexpr int NW = NW_;                            // waves per workgroup
  static constexpr int NT = 64 * NW;
  static constexpr int KS = KS_;                            // key tiles per ring stage, one per wave half
  static constexpr int RG = NW / KS;                        // row groups of 32 rows
  static constexpr int BQ = 32 * RG;                        // query rows per workgroup
  static constexpr int BK = kFwdBK;
  static constexpr int ROWS = BK * KS;                      // key rows per ring stage
  static constexpr int CA = DA / 8, CB = DB / 8;
  // key tiles in the row-padded layout (one operand base register) or swizzled
  static constexpr bool PAD = PAD_;
  static constexpr int SA = PAD ? PadRows<CA>::P : CA, SB = PAD ? PadRows<CB>::P : CB;   // slots per row
  static constexpr int STAGE = ROWS * (SA + SB);
  static constexpr int NSTAGE = NSTAGE_;
  // threads that stream the key tiles: the most (of 512, 384, 256, 128, 64, up to the workgroup) that split both
  // tensors' slots into whole loads
  static constexpr bool splits(int n) { return n <= NT && (ROWS * SA) % n == 0 && (ROWS * SB) % n == 0; }
  static constexpr int DMA_NT = splits(512) ? 512 : splits(384) ? 384 : splits(256) ? 256 : splits(128) ? 128 : 64;
  static constexpr int NCH = STAGE / DMA_NT;                // direct-to-LDS loads per streaming thread per tile
  static constexpr int MINB = MINB_;                        // workgroups per CU the registers are sized for
  // The second argument of __launch_bounds__ is waves per SIMD (execution
  // unit), not workgroups per CU: MINB workgroups of NW waves spread over the
  // four SIMDs of a CU.
  static constexpr int WAVES_PER_SIMD = (MINB * NW + 3) / 4;
  static_assert(DA % 64 == 0 && DB % 64 == 0, "head dims must be multiples of 64");
  static_assert(NSTAGE >= 2, "tile shape");
  static_assert(KS == 1 || KS == 2, "one or two key tiles per stage");
  static_assert(NW % KS == 0, "wave halves");
};

// Online pass of one workgroup over key tiles [t_begin, t_end) of the query
// rows q0 .. q0 + BQ - 1 of head bh; returns the lane's row state (both
// half-waves merged, and with KS = 2 both wave halves) and its row index in
// myq; owner: whether this wave writes the rows (the first wave half). tot:
// LDS for the per-lane totals of the chunked sums, NTOT * NT floats. With
// KS = 2, t_begin must be a multiple of 2 (the single pass starts at 0).
template <class C, bool CAUSAL, class Rows = SoftmaxRows>
__device__ __forceinline__ typename Rows::Partial fwd_pass(u32x4* st0, u32x4* st1, float* tot,
                                                           const uint16_t* __restrict__ Qa,
                                               const uint16_t* __restrict__ Ka, const uint16_t* __restrict__ Qb,
                                               const uint16_t* __restrict__ Kb, int NQ, int NK, int dra, int drb,
                                               float ca, float cb, int bh, int q0, int t_begin, int t_end,
                                               int& myq, bool& owner) {
  constexpr int DA = C::DA, DB = C::DB, BK = C::BK, KS = C::KS;
  static_assert(C::NSTAGE == 2, "the tile loop names two stage arrays");
  const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rg = wave % C::RG, kslot = wave / C::RG;   // row group, and which tile of a stage
  owner = kslot == 0;
  const int off = NK - NQ;
  const int qw = q0 + 32 * rg;
  myq = qw + (lane & 31);
  const int wlast = min(qw + 31, NQ - 1);

  int ntiles = (NK + BK - 1) / BK;
  if (CAUSAL) {
    const int kmax = min(q0 + C::BQ, NQ) - 1 + off;
    ntiles = kmax < 0 ? 0 : min(ntiles, kmax / BK + 1);
  }
  const WaveTiles wt = wave_tiles<CAUSAL>(qw, wlast, NQ, NK, ntiles);
  t_end = min(t_end, ntiles);
  const int u_begin = t_begin / KS, u_end = (t_end + KS - 1) / KS;   // ring stages
  const int kcm = CAUSAL ? myq + off : NK;

  bf16x8 qa[DA / 16], qb[DB / 16];
  load_q_operands<DA>(qa, Qa, (size_t)bh, NQ, myq, half, dra);
  load_q_operands<DB>(qb, Qb, (size_t)bh, NQ, myq, half, drb);

  const rsrc_t rka = make_rsrc(Ka + (size_t)bh * NK * dra, (uint32_t)NK * dra * 2u);
  const rsrc_t rkb = make_rsrc(Kb + (size_t)bh * NK * drb, (uint32_t)NK * drb * 2u);
  using Dma = typename std::conditional<C::PAD, PadTileDma<C::ROWS, C::CA, C::CB, C::DMA_NT>,
                                        TileDma<C::ROWS, C::CA, C::CB, C::DMA_NT>>::type;
  const bool streamer = wave < C::DMA_NT / 64;
  const Dma dma(streamer ? tid : 0, dra / 8, drb / 8);
  // operand bases of the row-padded layout (unused otherwise)
  const int base_a = C::PAD ? PadRows<C::CA>::base(lane & 31, half) : 0;
  const int base_b = C::PAD ? PadRows<C::CB>::base(lane & 31, half) : 0;
  // this wave's tile within a stage: rows kslot * BK .. of each tensor (both
  // layouts repeat their slot pattern every 16 rows)
  const int tile_a = kslot * BK * C::SA, tile_b = C::ROWS * C::SA + kslot * BK * C::SB;
  typename Rows::State st = Rows::init();
  bool have_total = false;   // uniform: whether tot holds a chunk yet

  if (u_begin < u_end && streamer) {
    dma.issue(rka, rkb, u_begin * C::ROWS, st0, wave, dra, drb);
    wait_vmem();   // stage u_begin
  }
  barrier_no_fence();
  // One stage: cur holds stage u, the next stage streams into nxt. The two
  // ring stages are separate arrays named by the loop (two stages per trip),
  // so the compiler can tell that a stage's reads never touch the stage being
  // loaded (and inserts no wait for those loads).
  auto step = [&](const u32x4* cur, u32x4* nxt, int u) {
    if (streamer) dma.issue(rka, rkb, (u + 1) * C::ROWS, nxt, wave, dra, drb);
    const int t = u * KS + kslot;   // this wave's key tile
    if (t <= wt.tlast && (KS == 1 || t < t_end)) {
      f32x16 sa, sb;
      fwd_logits<DA, DB, C::PAD>(cur + tile_a, cur + tile_b, qa, qb, sa, sb, lane, base_a, base_b);
      if (t >= wt.tmask) mask_tile(sa, sb, t * BK + 4 * half, NK, kcm);
      const bool ok = Rows::update(st, sa, sb, ca, cb, false);
      if (__builtin_amdgcn_ballot_w64(!ok) != 0) {   // uniform over the wave; rare
        // Form the logits again from the stage (still in LDS) rather than
        // keep the first ones live across the lazy pass (the barrier keeps
        // the compiler from reusing them); one operand read ahead keeps this
        // path within the register budget of four waves per SIMD.
        asm volatile("" ::: "memory");
        fwd_logits<DA, DB, C::PAD, 1>(cur + tile_a, cur + tile_b, qa, qb, sa, sb, lane, base_a, base_b);
        if (t >= wt.tmask) mask_tile(sa, sb, t * BK + 4 * half, NK, kcm);
        if (!ok) Rows::update(st, sa, sb, ca, cb, true);
      }
    }
    if ((u - u_begin) % kFoldTiles == kFoldTiles - 1 && u + 1 < u_end) {
      typename Rows::Partial r = Rows::partial(st, ca, cb);
      if (have_total) r = Rows::merge(Rows::load(tot, tid, C::NT), r);
      Rows::store(tot, tid, C::NT, r);
      have_total = true;
      Rows::reset(st);
    }
    wait_vmem();          // stage u + 1 has landed (for this wave) ...
    barrier_no_fence();   // ... and for every wave
  };
  for (int u = u_begin; u < u_end; u += 2) {
    step(st0, st1, u);
    if (u + 1 < u_end) step(st1, st0, u + 1);
  }
  wait_vmem();   // no load may still target LDS when the workgroup ends
  typename Rows::Partial mine = Rows::partial(st, ca, cb);
  if (have_total) mine = Rows::merge(Rows::load(tot, tid, C::NT), mine);
  mine = Rows::halfwave(mine);
  if constexpr (KS == 2) {
    // the second wave half hands its rows' states to the first through its
    // own total slots
    if (!owner) Rows::store(tot, tid, C::NT, mine);
    __syncthreads();
    if (owner) mine = Rows::merge(mine, Rows::load(tot, tid + 64 * C::RG, C::NT));
  }
  return mine;
}

// Whole key range per workgroup: grid B*H * ceil(N_Q / BQ).
template <class C, bool CAUSAL, bool PD = false>
__global__ void __launch_bounds__(C::NT, C::WAVES_PER_SIMD)
kl_fwd_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
              const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
              int NQ, int NK, int dra, int drb, float ca, float cb,
              float* __restrict__ kl, float* __restrict__ lse_a, float* __restrict__ lse_b) {
  // PD: the head dims may be padded (the rows in memory are dra, drb long);
  // otherwise they are the compile-time ones and the runtime values unused
  if constexpr (!PD) {
    dra = C::DA;
    drb = C::DB;
  }
  __shared__ u32x4 st0[C::STAGE];
  __shared__ u32x4 st1[C::STAGE];
  __shared__ float tot[SoftmaxRows::NTOT * C::NT];
  const int TQ = (NQ + C::BQ - 1) / C::BQ;
  int bh, qt;
  head_block<CAUSAL, C::MINB>(TQ, bh, qt);
  if (CAUSAL) qt = TQ - 1 - qt;   // rank 0: the last rows, the longest
  int myq;
  bool owner;
  const RowPartial p =
      fwd_pass<C, CAUSAL>(st0, st1, tot, Qa, Ka, Qb, Kb, NQ, NK, dra, drb, ca, cb, bh, qt * C::BQ, 0, 1 << 30,
                          myq, owner);
  if ((threadIdx.x & 32) == 0 && owner && myq < NQ) write_row(p, (size_t)bh * NQ + myq, kl, lse_a, lse_b);
}

// Forward of the sigmoid-score divergence (see SigmoidRows): the same tile
// loop over the whole key range, grid B*H * ceil(N_Q / BQ).
template <class C, bool CAUSAL, bool PD = false>
__global__ void __launch_bounds__(C::NT, C::WAVES_PER_SIMD)
kl_fwd_sigmoid_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                      const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                      int NQ, int NK, int dra, int drb, float ca, float cb,
                      float* __restrict__ kl, float* __restrict__ mass_a, float* __restrict__ mass_b) {
  // PD: the head dims may be padded (the rows in memory are dra, drb long);
  // otherwise they are the compile-time ones and the runtime values unused
  if constexpr (!PD) {
    dra = C::DA;
    drb = C::DB;
  }
  __shared__ u32x4 st0[C::STAGE];
  __shared__ u32x4 st1[C::STAGE];
  __shared__ float tot[SigmoidRows::NTOT * C::NT];
  const int TQ = (NQ + C::BQ - 1) / C::BQ;
  int bh, qt;
  head_block<CAUSAL, C::MINB>(TQ, bh, qt);
  if (CAUSAL) qt = TQ - 1 - qt;   // rank 0: the last rows, the longest
  int myq;
  bool owner;
  const SigmoidPartial p = fwd_pass<C, CAUSAL, SigmoidRows>(st0, st1, tot, Qa, Ka, Qb, Kb, NQ, NK, dra, drb, ca, cb,
                                                            bh, qt * C::BQ, 0, 1 << 30, myq, owner);
  if ((threadIdx.x & 32) == 0 && owner && myq < NQ) write_row_sigmoid(p, (size_t)bh * NQ + myq, kl, mass_a, mass_b);
}

// Split-K partial pass (Sec. 3.3): grid B*H * ceil(N_Q / BQ) * W; workgroup
// (head, query tile, w) covers key tiles [w * chunk, (w + 1) * chunk) and
// writes the five row statistics to part[k][w][B*H*N_Q], k = (m_a, l_a, m_b,
// l_b, acc), maxima in the base-2 domain.
template <class C, bool CAUSAL, bool PD = false>
__global__ void __launch_bounds__(C::NT, C::WAVES_PER_SIMD)
kl_fwd_partial_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                      const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                      int NQ, int NK, int dra, int drb, float ca, float cb, int W, int chunk, float* __restrict__ part) {
  // PD: the head dims may be padded (the rows in memory are dra, drb long);
  // otherwise they are the compile-time ones and the runtime values unused
  if constexpr (!PD) {
    dra = C::DA;
    drb = C::DB;
  }
  __shared__ u32x4 st0[C::STAGE];
  __shared__ u32x4 st1[C::STAGE];
  __shared__ float tot[SoftmaxRows::NTOT * C::NT];
  const int TQ = (NQ + C::BQ - 1) / C::BQ;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int w = logical % W;
  const int rest = logical / W;
  const int bh = rest / TQ;
  const int qt = rest - bh * TQ;
  static_assert(C::KS == 1, "chunks of single key tiles");
  int myq;
  bool owner;
  const RowPartial p = fwd_pass<C, CAUSAL>(st0, st1, tot, Qa, Ka, Qb, Kb, NQ, NK, dra, drb, ca, cb, bh, qt * C::BQ,
                                           w * chunk, (w + 1) * chunk, myq, owner);
  if ((threadIdx.x & 32) == 0 && myq < NQ) {
    const size_t rows = (size_t)gridDim.x / W / TQ * NQ;   // B*H*N_Q
    const size_t ri = (size_t)w * rows + (size_t)bh * NQ + myq;
    const size_t plane = (size_t)W * rows;
    part[ri] = p.ma;
    part[ri + plane] = p.la;
    part[ri + 2 * plane] = p.mb;
    part[ri + 3 * plane] = p.lb;
    part[ri + 4 * plane] = p.acc;
  }
}

// Split-K reduce (Sec. 3.3): one wave per row. Lane w merges partials w,
// w + 64, ... (independent loads, all in flight together), then the wave
// merges its 64 lane states by a butterfly of shuffles, and lane 0 writes
// KL, LSE_a, LSE_b. One thread per row walking its W partials in sequence
// spent a load latency per partial: 14-20 us at W = 32.
constexpr int kMergeRowsPerBlock = 4;
static __global__ void __launch_bounds__(64 * kMergeRowsPerBlock)
kl_fwd_merge_kernel(const float* __restrict__ part, int W, size_t rows, float* __restrict__ kl,
                    float* __restrict__ lse_a, float* __restrict__ lse_b) {
  const int lane = threadIdx.x & 63;
  const size_t ri = (size_t)blockIdx.x * kMergeRowsPerBlock + (threadIdx.x >> 6);
  if (ri >= rows) return;   // whole waves leave together
  const size_t plane = (size_t)W * rows;
  RowPartial acc{kNegInf, 0.f, kNegInf, 0.f, 0.f};
  for (int w = lane; w < W; w += 64) {
    const size_t i = (size_t)w * rows + ri;
    acc = merge_partials(acc, RowPartial{part[i], part[i + plane], part[i + 2 * plane], part[i + 3 * plane],
                                         part[i + 4 * plane]});
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const RowPartial other{__shfl_xor(acc.ma, off), __shfl_xor(acc.la, off), __shfl_xor(acc.mb, off),
                           __shfl_xor(acc.lb, off), __shfl_xor(acc.acc, off)};
    acc = merge_partials(acc, other);
  }
  if (lane == 0) write_row(acc, ri, kl, lse_a, lse_b);
}

// Configuration per head-dim pair: eight waves (256 rows share each key
// tile) and a two-stage ring. Two workgroups per CU (four waves per SIMD)
// need the whole kernel in 128 registers per lane: the pairs up to d1 + d2 =
// 192 and (128, 128) compile to at most 128 without spilling, (64, 192) and
// (192, 64) need 136 and keep one workgroup per CU. Wider heads take four
// waves and one workgroup. The launch bounds hold the compiler to these
// occupancies; tests/test_build_resources.py checks them on the compiled code.
template <int DA, int DB>
constexpr bool kFwdTwoPerCu = (DA + DB <= 192) || (DA == 128 && DB == 128);
template <int DA, int DB>
using FwdCfg = typename std::conditional<(DA + DB <= 256), FwdTraits<DA, DB, 2, kFwdTwoPerCu<DA, DB> ? 2 : 1, 8, true>,
                                         FwdTraits<DA, DB, 2, 1, 4, true>>::type;

// Causal heads with few 256-row blocks (the launcher's rule): four waves in
// the default key-tile layout, two workgroups per CU.
template <int DA, int DB>
using FwdCausalSmallCfg = FwdTraits<DA, DB, 2, 2, 4, true>;

// Causal grids of those that fit one round of resident workgroups (d1 + d2 <=
// 192): the same 128 rows per workgroup as eight waves in two halves that
// take alternate key tiles (two tiles per ring stage, swizzled layout: the
// padded one would not leave room for two workgroups per CU). With every
// workgroup resident at once the longest causal block sets the time, and the
// two halves split it. Wider pairs do not fit this in 128 registers.
template <int DA, int DB>
using FwdCausalKeySplitCfg = FwdTraits<DA, DB, 2, 2, 8, false, 2>;

// Padded head dims (32, 96, 160, 224 run as 64, 128, 192, 256): one
// configuration for every shape, four waves and 128 rows per workgroup.
template <int DA, int DB>
using FwdPadDimCfg = FwdTraits<DA, DB, 2, (DA + DB <= 256) ? 2 : 1, 4, true>;

// Few query rows per head (decode-like shapes): NW waves per workgroup; four
// one-wave or two four-wave workgroups per CU (one for wide heads).
template <int DA, int DB, int NW>
using FwdSmallCfg = FwdTraits<DA, DB, 2, (DA + DB <= 256) ? (NW == 1 ? 4 : 2) : 1, NW>;

// Which configuration a head shape takes (the launch units instantiate
// them): one wave for at most 32 query rows, four waves for at most 128
// (d1 + d2 <= 256), the 128-row causal configurations when 256-row
// workgroups would number fewer than four per CU, otherwise FwdCfg. The
// causal 128-row configuration measured 10-16% faster on such shapes (twice
// the workgroups: the two waves sharing a SIMD come from different workgroups
// and the long causal rows spread over more CUs); non-causal shapes of the
// same size were 4-6% slower with it and keep the default. Of those causal
// grids, the ones that fit one round (at most 512 workgroups of 128 rows, d1 +
// d2 <= 192) take the key-split configuration: 7-10% faster there, about 1%
// slower on two-round grids.
enum class FwdShape { kOneWave, kFourWaves, kCausalSmall, kCausalKeySplit, kDefault };
constexpr long long kCausalSmallGrid = 1024;
constexpr long long kCausalOneRound = 512;
inline FwdShape fwd_shape(int da, int db, int n_q, long long bh, bool causal) {
  if (n_q <= 32) return FwdShape::kOneWave;
  if (da + db <= 256) {
    if (n_q <= 128) return FwdShape::kFourWaves;
    if (causal && bh * ((n_q + 255) / 256) < kCausalSmallGrid) {
      if (da + db <= 192 && bh * ((n_q + 127) / 128) <= kCausalOneRound) return FwdShape::kCausalKeySplit;
      return FwdShape::kCausalSmall;
    }
  }
  return FwdShape::kDefault;
}

}  // namespace streamkl
