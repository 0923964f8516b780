// Forward kernel of the fused attention-KL (Algorithm 1, Sec. 3.2).
//
// One workgroup owns BQ = 128 query rows of one (batch, head): each of its
// four waves keeps 32 rows of Q_a and Q_b in registers as MFMA B operands and
// the workgroup streams key tiles K_a, K_b (BK rows) through a two-stage LDS
// ring. Per tile each wave forms S_a^T = K_a Q_a^T and S_b^T = K_b Q_b^T on
// the 32x32x16 bf16 MFMA with fp32 accumulation. In the transposed result a
// lane owns one query row (column l % 32) and 16 keys per 32-key block, so
// every row reduction is in-lane: the two half-waves (l / 32 = 0, 1) hold
// disjoint key subsets of the same rows and each keeps its own five running
// scalars (m_a, l_a, m_b, l_b, acc), merged once at the end by the split-K
// rule of Sec. 3.3. Nothing crosses lanes inside the key loop.
//
// Arithmetic is in the base-2 domain (Sec. 5 uses exp2): t = raw * s * log2(e),
// p = 2^(t - m), and acc = sum p_a (t_a - t_b) (eq:acc-invariant in base 2,
// so acc * ln 2 is the paper's acc). Per element: one max (as max3 pairs), one
// fma and one exp2 per distribution, two adds and a sub + fma for acc.
// Causal key tiles past a row block's frontier are never loaded; only tiles
// that cross the diagonal or the ragged key tail take the masked path.
//
// "a" is the distribution in the first KL slot, "b" the second: the host
// passes (Q1,K1) as a for KL(P1||P2) and swaps the roles for KL(P2||P1).
#pragma once

#include "kl_common.hpp"

namespace streamkl {

// Tile configuration of the forward kernel.
//   BK      key rows per tile (a multiple of 32)
//   NSTAGE  depth of the LDS ring of key tiles
//   PIPE    software pipeline: the MFMAs of tile kt + 1 are issued among the
//           vector instructions of tile kt's online update
//   MINB    workgroups per CU the register budget is sized for
//   BATCH   issue all LDS operand reads of a 32-key block before its MFMAs
template <int DA_, int DB_, int BK_, int NSTAGE_, bool PIPE_, int MINB_, bool BATCH_ = false>
struct FwdTraits {
  static constexpr int DA = DA_, DB = DB_;
  static constexpr int NW = 4;                              // waves per workgroup
  static constexpr int BQ = 32 * NW;                        // query rows per workgroup
  static constexpr int BK = BK_;
  static constexpr int NMB = BK / 32;                       // 32-key MFMA blocks per tile
  static constexpr int CA = DA / 8, CB = DB / 8;            // 16-byte chunks per row
  static constexpr int STAGE = BK * (CA + CB);              // chunks per LDS stage
  static constexpr int NSTAGE = NSTAGE_;
  static constexpr int NCH = STAGE / kThreads;              // direct-to-LDS loads per thread per tile
  static constexpr bool PIPE = PIPE_;
  static constexpr int MINB = MINB_;
  static constexpr bool BATCH = BATCH_;
  static_assert(DA % 64 == 0 && DB % 64 == 0, "head dims must be multiples of 64");
  static_assert(BK % 32 == 0 && NSTAGE >= 2, "tile shape");
};

// The configuration used for every head-dim pair: 32-key tiles, a two-stage
// ring, no software pipeline (on gfx950 a wave's own MFMAs and vector work
// serialise, so overlap comes from the other resident waves instead).
template <int DA, int DB>
using FwdCfg = FwdTraits<DA, DB, 32, 2, false, (DA + DB <= 256) ? 2 : 1>;

// Five running row scalars of one half-wave (base-2 domain, see above).
struct RowState {
  float ma, la, mb, lb, acc;
};

template <class C, bool MASK>
__device__ __forceinline__ void fwd_tile_update(RowState& st, const f32x16 (&sa)[C::NMB], const f32x16 (&sb)[C::NMB],
                                                float ca, float cb, int kbase, int klimit_excl,
                                                int kcausal_max) {
  constexpr int NMB = C::NMB;
  // kbase: key index of register 0 of block 0 for this lane (k0 + 4 * half).
  // A key k is allowed iff k < klimit_excl and k <= kcausal_max.
  float ra[NMB][16], rb[NMB][16];
  bool ok[NMB][16];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int k = kbase + 32 * mb + 8 * (i >> 2) + (i & 3);
      ok[mb][i] = MASK ? (k < klimit_excl && k <= kcausal_max) : true;
      ra[mb][i] = ok[mb][i] ? sa[mb][i] : kNegInf;
      rb[mb][i] = ok[mb][i] ? sb[mb][i] : kNegInf;
    }
  // tile row maxima of the raw dot products (s > 0, so the scaled max is c * max)
  float xa0 = ra[0][0], xa1 = ra[0][1], xb0 = rb[0][0], xb1 = rb[0][1];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int i = (mb == 0 ? 2 : 0); i < 16; i += 2) {
      xa0 = fmaxf(xa0, ra[mb][i]);
      xa1 = fmaxf(xa1, ra[mb][i + 1]);
      xb0 = fmaxf(xb0, rb[mb][i]);
      xb1 = fmaxf(xb1, rb[mb][i + 1]);
    }
  const float ma_new = fmaxf(st.ma, fmaxf(xa0, xa1) * ca);
  const float mb_new = fmaxf(st.mb, fmaxf(xb0, xb1) * cb);
  // a half-wave that has seen only masked keys keeps m = -inf; use 0 as the
  // reference so that 2^(t - m) and the correction factors stay NaN-free.
  const float ua = (MASK && ma_new == kNegInf) ? 0.f : ma_new;
  const float ub = (MASK && mb_new == kNegInf) ? 0.f : mb_new;
  const float alpha_a = exp2_fast(st.ma - ua);
  const float alpha_b = exp2_fast(st.mb - ub);
  float sla[2] = {0.f, 0.f}, slb[2] = {0.f, 0.f}, sac[2] = {0.f, 0.f};
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float xa = __builtin_fmaf(ra[mb][i], ca, -ua);
      const float xb = __builtin_fmaf(rb[mb][i], cb, -ub);
      const float pa = exp2_fast(xa);
      const float pb = exp2_fast(xb);
      sla[i & 1] += pa;
      slb[i & 1] += pb;
      const float term = pa * (xa - xb);
      sac[i & 1] += MASK ? (ok[mb][i] ? term : 0.f) : term;
    }
  const float tla = sla[0] + sla[1];
  st.la = __builtin_fmaf(alpha_a, st.la, tla);
  st.lb = __builtin_fmaf(alpha_b, st.lb, slb[0] + slb[1]);
  // sum p_a (t_a - t_b) = sum p_a (x_a - x_b) + (m_a - m_b) sum p_a
  st.acc = __builtin_fmaf(alpha_a, st.acc, __builtin_fmaf(ua - ub, tla, sac[0] + sac[1]));
  st.ma = ma_new;
  st.mb = mb_new;
}

// S^T tiles of one key tile (all 32-key blocks) on the MFMA: A = key rows from
// LDS, B = the lane's resident query rows; the two accumulation chains
// alternate. With C::BATCH all operand reads of a block are issued before its
// first MFMA (a scheduling barrier keeps the compiler from pairing each read
// with its MFMA, which exposes the LDS latency on every step, at the price of
// 4 VGPRs per operand).
template <class C>
__device__ __forceinline__ void fwd_logits(const u32x4* stage, const bf16x8 (&qa)[C::DA / 16],
                                           const bf16x8 (&qb)[C::DB / 16], f32x16 (&sa)[C::NMB],
                                           f32x16 (&sb)[C::NMB], int lane) {
  constexpr int KA = C::DA / 16, KB = C::DB / 16, KM = KA > KB ? KA : KB;
  const int half = lane >> 5;
  const u32x4* ta = stage;
  const u32x4* tb = stage + C::BK * C::CA;
#pragma unroll
  for (int mb = 0; mb < C::NMB; ++mb) {
    const int r = 32 * mb + (lane & 31);
    bf16x8 oa[KA], ob[KB];
#pragma unroll
    for (int ks = 0; ks < KM; ++ks) {
      if (ks < KA) oa[ks] = lds_row8<C::CA>(ta, r, 2 * ks + half);
      if (ks < KB) ob[ks] = lds_row8<C::CB>(tb, r, 2 * ks + half);
    }
    if constexpr (C::BATCH) __builtin_amdgcn_sched_barrier(0);
    f32x16 acc_a = zero16(), acc_b = zero16();
#pragma unroll
    for (int ks = 0; ks < KM; ++ks) {
      if (ks < KA) acc_a = mfma32(oa[ks], qa[ks], acc_a);
      if (ks < KB) acc_b = mfma32(ob[ks], qb[ks], acc_b);
    }
    sa[mb] = acc_a;
    sb[mb] = acc_b;
  }
}

// Scheduling hint for one pipelined step: spread the NM MFMAs (and their LDS
// operand reads) of the next tile evenly over the NV vector instructions of
// the current tile's online update.
template <int NM, int NV>
__device__ __forceinline__ void interleave_mfma_valu() {
  constexpr int per = (NV + NM - 1) / NM;
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);      // operand reads run ahead
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // one LDS read
    __builtin_amdgcn_sched_group_barrier(0x402, per, 0);  // VALU and transcendental
  }
}

// One step of a wave: online update of the current tile's logits (sa, sb)
// and, if NEXT, formation of the next tile's logits (na, nb) alongside.
template <class C, bool MASK, bool NEXT>
__device__ __forceinline__ void fwd_step(RowState& st, const f32x16 (&sa)[C::NMB], const f32x16 (&sb)[C::NMB],
                                         const u32x4* next, const bf16x8 (&qa)[C::DA / 16],
                                         const bf16x8 (&qb)[C::DB / 16], f32x16 (&na)[C::NMB],
                                         f32x16 (&nb)[C::NMB], float ca, float cb, int kbase, int NK,
                                         int kcausal_max, int lane) {
  if constexpr (NEXT) fwd_logits<C>(next, qa, qb, na, nb, lane);
  fwd_tile_update<C, MASK>(st, sa, sb, ca, cb, kbase, NK, kcausal_max);
  if constexpr (NEXT) interleave_mfma_valu<C::NMB * (C::DA + C::DB) / 16, C::NMB * (MASK ? 240 : 160)>();
}

template <class C, bool CAUSAL>
__global__ void __launch_bounds__(kThreads, C::MINB)
kl_fwd_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
              const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
              int NQ, int NK, float ca, float cb,
              float* __restrict__ kl, float* __restrict__ lse_a, float* __restrict__ lse_b) {
  constexpr int DA = C::DA, DB = C::DB, R = C::NSTAGE;
  __shared__ u32x4 smem[R * C::STAGE];   // ring of key tiles: tile t lives in stage t % R

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int TQ = (NQ + C::BQ - 1) / C::BQ;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int bh = logical / TQ;
  int qt = logical - bh * TQ;
  if (CAUSAL) qt = TQ - 1 - qt;   // longest rows first
  const int q0 = qt * C::BQ;
  const int off = NK - NQ;        // bottom-right alignment: row i sees keys <= i + off
  const int qw = q0 + 32 * wave;  // first row of this wave
  const int myq = qw + (lane & 31);
  const int wlast = min(qw + 31, NQ - 1);   // last valid row of this wave

  int ntiles = (NK + C::BK - 1) / C::BK;
  if (CAUSAL) {
    const int kmax = min(q0 + C::BQ, NQ) - 1 + off;
    ntiles = kmax < 0 ? 0 : min(ntiles, kmax / C::BK + 1);
  }

  // Q rows of this lane as MFMA B operands: chunk 2 * ks + half of row myq.
  bf16x8 qa[DA / 16], qb[DB / 16];
  {
    const bool okq = myq < NQ;
    const u32x4* pa = reinterpret_cast<const u32x4*>(Qa + ((size_t)bh * NQ + (okq ? myq : 0)) * DA);
    const u32x4* pb = reinterpret_cast<const u32x4*>(Qb + ((size_t)bh * NQ + (okq ? myq : 0)) * DB);
#pragma unroll
    for (int ks = 0; ks < DA / 16; ++ks)
      qa[ks] = __builtin_bit_cast(bf16x8, okq ? pa[2 * ks + half] : u32x4{0u, 0u, 0u, 0u});
#pragma unroll
    for (int ks = 0; ks < DB / 16; ++ks)
      qb[ks] = __builtin_bit_cast(bf16x8, okq ? pb[2 * ks + half] : u32x4{0u, 0u, 0u, 0u});
  }

  const rsrc_t rka = make_rsrc(Ka + (size_t)bh * NK * DA, (uint32_t)NK * DA * 2u);
  const rsrc_t rkb = make_rsrc(Kb + (size_t)bh * NK * DB, (uint32_t)NK * DB * 2u);
  const TileDma<C::BK, C::CA, C::CB> dma(tid);
  RowState st{kNegInf, 0.f, kNegInf, 0.f, 0.f};
  const int kcm = CAUSAL ? myq + off : NK;
  auto stage_of = [&](int t) { return smem + (t % R) * C::STAGE; };

  // A wave has work in key tile kt while kt is not past its causal frontier;
  // once inactive it stays inactive for every later tile.
  auto active = [&](int kt) { return qw < NQ && (!CAUSAL || kt * C::BK <= wlast + off); };
  auto masked = [&](int kt) {
    return kt * C::BK + C::BK > NK || (CAUSAL && kt * C::BK + C::BK - 1 > qw + off);
  };

  if constexpr (C::PIPE) {
    // Iteration kt runs the online update of tile kt's logits while the MFMA
    // forms tile kt + 1's logits from its LDS stage, and tile kt + R streams
    // into the stage tile kt occupied (its logits were formed one iteration
    // earlier). Every iteration issues exactly one tile of loads (past the end
    // they only fill zeros), so after tile kt + 2 has landed the loads still
    // in flight are the constant (R - 2) tiles.
    f32x16 s0a[C::NMB], s0b[C::NMB], s1a[C::NMB], s1b[C::NMB];
    auto step = [&](int kt, const f32x16 (&ca_)[C::NMB], const f32x16 (&cb_)[C::NMB], f32x16 (&na)[C::NMB],
                    f32x16 (&nb)[C::NMB]) {
      dma.issue(rka, rkb, (kt + R) * C::BK, stage_of(kt), wave);
      if (active(kt)) {
        const bool nxt = kt + 1 < ntiles && active(kt + 1);
        const int kbase = kt * C::BK + 4 * half;
        const u32x4* ns = stage_of(kt + 1);
        if (masked(kt)) {
          if (nxt) fwd_step<C, true, true>(st, ca_, cb_, ns, qa, qb, na, nb, ca, cb, kbase, NK, kcm, lane);
          else fwd_step<C, true, false>(st, ca_, cb_, ns, qa, qb, na, nb, ca, cb, kbase, NK, kcm, lane);
        } else {
          if (nxt) fwd_step<C, false, true>(st, ca_, cb_, ns, qa, qb, na, nb, ca, cb, kbase, NK, NK, lane);
          else fwd_step<C, false, false>(st, ca_, cb_, ns, qa, qb, na, nb, ca, cb, kbase, NK, NK, lane);
        }
      }
      wait_vmem_le<(R - 2) * C::NCH>();   // tile kt + 2 has landed (for this wave) ...
      __syncthreads();                    // ... and for every wave
    };
    if (ntiles > 0) {
#pragma unroll
      for (int t = 0; t < R; ++t) dma.issue(rka, rkb, t * C::BK, smem + t * C::STAGE, wave);
      wait_vmem_le<(R - 1) * C::NCH>();   // tile 0
      __syncthreads();
      if (active(0)) fwd_logits<C>(smem, qa, qb, s0a, s0b, lane);
      wait_vmem_le<(R - 2) * C::NCH>();   // tile 1
      __syncthreads();
    }
    for (int kt = 0; kt < ntiles; kt += 2) {
      step(kt, s0a, s0b, s1a, s1b);
      if (kt + 1 < ntiles) step(kt + 1, s1a, s1b, s0a, s0b);
    }
  } else {
    // Iteration kt forms and reduces tile kt from its stage while tile
    // kt + R - 1 streams into the stage tile kt - 1 occupied; after tile kt + 1
    // has landed, (R - 2) tiles of loads are still in flight.
    if (ntiles > 0) {
#pragma unroll
      for (int t = 0; t < R - 1; ++t) dma.issue(rka, rkb, t * C::BK, smem + t * C::STAGE, wave);
      wait_vmem_le<(R - 2) * C::NCH>();   // tile 0
    }
    __syncthreads();
    for (int kt = 0; kt < ntiles; ++kt) {
      dma.issue(rka, rkb, (kt + R - 1) * C::BK, stage_of(kt + R - 1), wave);
      if (active(kt)) {
        f32x16 sa[C::NMB], sb[C::NMB];
        fwd_logits<C>(stage_of(kt), qa, qb, sa, sb, lane);
        const int kbase = kt * C::BK + 4 * half;
        if (masked(kt)) fwd_tile_update<C, true>(st, sa, sb, ca, cb, kbase, NK, kcm);
        else fwd_tile_update<C, false>(st, sa, sb, ca, cb, kbase, NK, NK);
      }
      wait_vmem_le<(R - 2) * C::NCH>();   // tile kt + 1 has landed (for this wave) ...
      __syncthreads();                    // ... and for every wave
    }
  }

  // Merge the two half-waves of each row (split-K merge of Sec. 3.3).
  RowState o;
  o.ma = __shfl_xor(st.ma, 32);
  o.la = __shfl_xor(st.la, 32);
  o.mb = __shfl_xor(st.mb, 32);
  o.lb = __shfl_xor(st.lb, 32);
  o.acc = __shfl_xor(st.acc, 32);
  if (half == 0 && myq < NQ) {
    const float ma = fmaxf(st.ma, o.ma), mb = fmaxf(st.mb, o.mb);
    float out_kl = 0.f, out_la = kNegInf, out_lb = kNegInf;
    if (ma != kNegInf) {
      const float f0 = exp2_fast(st.ma - ma), f1 = exp2_fast(o.ma - ma);
      const float g0 = exp2_fast(st.mb - mb), g1 = exp2_fast(o.mb - mb);
      const float la = st.la * f0 + o.la * f1;
      const float lb = st.lb * g0 + o.lb * g1;
      const float acc = st.acc * f0 + o.acc * f1;
      out_la = (ma + log2f(la)) * kLn2;       // LSE_t = m_t + ln l_t (natural log)
      out_lb = (mb + log2f(lb)) * kLn2;
      out_kl = acc * kLn2 / la + out_lb - out_la;   // eq:kl-final
    }
    const size_t ri = (size_t)bh * NQ + myq;
    kl[ri] = out_kl;
    lse_a[ri] = out_la;
    lse_b[ri] = out_lb;
  }
}

// ----------------------------------------------------------------------------
// Ping-pong forward. On gfx950 a wave that interleaves MFMAs with its own
// vector work serialises the two, while an MFMA-only wave and a vector-only
// wave sharing a SIMD run side by side. So the workgroup holds two groups of
// four waves, one wave of each group per SIMD, and every key tile takes two
// half-steps separated by workgroup barriers: in one half-step group 0 forms
// the tile's logits on the MFMA while group 1 runs the online update of the
// previous tile, in the next half-step the roles swap. Each wave keeps a
// single logit tile in registers. Rows are interleaved between the groups
// (32-row blocks alternate) so that causal frontiers stay balanced.
// ----------------------------------------------------------------------------
template <int DA_, int DB_, int BK_, int NSTAGE_>
struct FwdPPTraits {
  static constexpr int DA = DA_, DB = DB_;
  static constexpr int NW = 8;                              // waves per workgroup (two groups of four)
  static constexpr int NT = 64 * NW;
  static constexpr int BQ = 32 * NW;                        // query rows per workgroup
  static constexpr int BK = BK_;
  static constexpr int NMB = BK / 32;
  static constexpr int CA = DA / 8, CB = DB / 8;
  static constexpr int STAGE = BK * (CA + CB);
  static constexpr int NSTAGE = NSTAGE_;
  static constexpr int NCH = STAGE / NT;
  static constexpr bool PIPE = false;
  static constexpr int MINB = 1;
  static constexpr bool BATCH = true;
  static_assert(DA % 64 == 0 && DB % 64 == 0, "head dims must be multiples of 64");
  static_assert(BK % 32 == 0 && NSTAGE >= 2 && STAGE % NT == 0, "tile shape");
};

template <class C, bool CAUSAL>
__global__ void __launch_bounds__(C::NT, 1)
kl_fwd_pp_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                 const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                 int NQ, int NK, float ca, float cb,
                 float* __restrict__ kl, float* __restrict__ lse_a, float* __restrict__ lse_b) {
  constexpr int DA = C::DA, DB = C::DB, R = C::NSTAGE;
  __shared__ u32x4 smem[R * C::STAGE];   // ring of key tiles: tile t lives in stage t % R

  const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;               // 0: logits first, 1: update first
  const int TQ = (NQ + C::BQ - 1) / C::BQ;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int bh = logical / TQ;
  int qt = logical - bh * TQ;
  if (CAUSAL) qt = TQ - 1 - qt;   // longest rows first
  const int q0 = qt * C::BQ;
  const int off = NK - NQ;
  const int qw = q0 + 32 * (2 * (wave & 3) + grp);   // 32-row blocks alternate between the groups
  const int myq = qw + (lane & 31);
  const int wlast = min(qw + 31, NQ - 1);

  int ntiles = (NK + C::BK - 1) / C::BK;
  if (CAUSAL) {
    const int kmax = min(q0 + C::BQ, NQ) - 1 + off;
    ntiles = kmax < 0 ? 0 : min(ntiles, kmax / C::BK + 1);
  }

  bf16x8 qa[DA / 16], qb[DB / 16];
  {
    const bool okq = myq < NQ;
    const u32x4* pa = reinterpret_cast<const u32x4*>(Qa + ((size_t)bh * NQ + (okq ? myq : 0)) * DA);
    const u32x4* pb = reinterpret_cast<const u32x4*>(Qb + ((size_t)bh * NQ + (okq ? myq : 0)) * DB);
#pragma unroll
    for (int ks = 0; ks < DA / 16; ++ks)
      qa[ks] = __builtin_bit_cast(bf16x8, okq ? pa[2 * ks + half] : u32x4{0u, 0u, 0u, 0u});
#pragma unroll
    for (int ks = 0; ks < DB / 16; ++ks)
      qb[ks] = __builtin_bit_cast(bf16x8, okq ? pb[2 * ks + half] : u32x4{0u, 0u, 0u, 0u});
  }

  const rsrc_t rka = make_rsrc(Ka + (size_t)bh * NK * DA, (uint32_t)NK * DA * 2u);
  const rsrc_t rkb = make_rsrc(Kb + (size_t)bh * NK * DB, (uint32_t)NK * DB * 2u);
  const TileDma<C::BK, C::CA, C::CB, C::NT> dma(tid);
  RowState st{kNegInf, 0.f, kNegInf, 0.f, 0.f};
  const int kcm = CAUSAL ? myq + off : NK;
  auto stage_of = [&](int t) { return smem + (t % R) * C::STAGE; };
  auto active = [&](int kt) { return kt >= 0 && qw < NQ && (!CAUSAL || kt * C::BK <= wlast + off); };
  auto masked = [&](int kt) {
    return kt * C::BK + C::BK > NK || (CAUSAL && kt * C::BK + C::BK - 1 > qw + off);
  };
  f32x16 sa[C::NMB], sb[C::NMB];
  auto logits = [&](int kt) {
    if (active(kt)) fwd_logits<C>(stage_of(kt), qa, qb, sa, sb, lane);
  };
  auto update = [&](int kt) {
    if (active(kt)) {
      const int kbase = kt * C::BK + 4 * half;
      if (masked(kt)) fwd_tile_update<C, true>(st, sa, sb, ca, cb, kbase, NK, kcm);
      else fwd_tile_update<C, false>(st, sa, sb, ca, cb, kbase, NK, NK);
    }
  };

  // Tile kt + R - 1 streams into the stage of tile kt - 1 (both groups have
  // formed its logits); after tile kt + 1 has landed, (R - 2) tiles of loads
  // are still in flight.
  if (ntiles > 0) {
#pragma unroll
    for (int t = 0; t < R - 1; ++t) dma.issue(rka, rkb, t * C::BK, smem + t * C::STAGE, wave);
    wait_vmem_le<(R - 2) * C::NCH>();
  }
  __syncthreads();
  for (int kt = 0; kt < ntiles; ++kt) {
    dma.issue(rka, rkb, (kt + R - 1) * C::BK, stage_of(kt + R - 1), wave);
    if (grp == 0) logits(kt);
    else update(kt - 1);
    __syncthreads();
    if (grp == 0) update(kt);
    else logits(kt);
    wait_vmem_le<(R - 2) * C::NCH>();
    __syncthreads();
  }
  if (grp == 1) update(ntiles - 1);

  RowState o;
  o.ma = __shfl_xor(st.ma, 32);
  o.la = __shfl_xor(st.la, 32);
  o.mb = __shfl_xor(st.mb, 32);
  o.lb = __shfl_xor(st.lb, 32);
  o.acc = __shfl_xor(st.acc, 32);
  if (half == 0 && myq < NQ) {
    const float ma = fmaxf(st.ma, o.ma), mb = fmaxf(st.mb, o.mb);
    float out_kl = 0.f, out_la = kNegInf, out_lb = kNegInf;
    if (ma != kNegInf) {
      const float f0 = exp2_fast(st.ma - ma), f1 = exp2_fast(o.ma - ma);
      const float g0 = exp2_fast(st.mb - mb), g1 = exp2_fast(o.mb - mb);
      const float la = st.la * f0 + o.la * f1;
      const float lb = st.lb * g0 + o.lb * g1;
      const float acc = st.acc * f0 + o.acc * f1;
      out_la = (ma + log2f(la)) * kLn2;
      out_lb = (mb + log2f(lb)) * kLn2;
      out_kl = acc * kLn2 / la + out_lb - out_la;
    }
    const size_t ri = (size_t)bh * NQ + myq;
    kl[ri] = out_kl;
    lse_a[ri] = out_la;
    lse_b[ri] = out_lb;
  }
}

}  // namespace streamkl
