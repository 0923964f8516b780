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

template <int DA, int DB>
struct FwdCfg {
  static constexpr int NW = 4;                              // waves per workgroup
  static constexpr int BQ = 32 * NW;                        // query rows per workgroup
  static constexpr int BK = (DA + DB <= 256) ? 64 : 32;     // key rows per tile
  static constexpr int NMB = BK / 32;                       // 32-key MFMA blocks per tile
  static constexpr int CA = DA / 8, CB = DB / 8;            // 16-byte chunks per row
  static constexpr int STAGE = BK * (CA + CB);              // chunks per LDS stage
  static constexpr int MINB = (DA + DB <= 256) ? 2 : 1;     // workgroups per CU to fit
  static_assert(DA % 64 == 0 && DB % 64 == 0, "head dims must be multiples of 64");
};

// Five running row scalars of one half-wave (base-2 domain, see above).
struct RowState {
  float ma, la, mb, lb, acc;
};

template <int DA, int DB, bool MASK>
__device__ __forceinline__ void fwd_tile_update(RowState& st, const f32x16 (&sa)[FwdCfg<DA, DB>::NMB],
                                                const f32x16 (&sb)[FwdCfg<DA, DB>::NMB],
                                                float ca, float cb, int kbase, int klimit_excl,
                                                int kcausal_max) {
  constexpr int NMB = FwdCfg<DA, DB>::NMB;
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

// One key tile of one wave: S^T tiles on the MFMA, then the online update.
template <int DA, int DB, bool CAUSAL>
__device__ __forceinline__ void fwd_tile(const u32x4* stage, const bf16x8 (&qa)[DA / 16], const bf16x8 (&qb)[DB / 16],
                                         RowState& st, int k0, int NK, int qw, int wlast, int off, int myq,
                                         float ca, float cb, int lane) {
  using C = FwdCfg<DA, DB>;
  bool active = qw <= wlast;
  bool need_mask = k0 + C::BK > NK;
  if (CAUSAL) {
    active = active && (k0 <= wlast + off);
    need_mask = need_mask || (k0 + C::BK - 1 > qw + off);
  }
  if (!active) return;
  const int half = lane >> 5;
  const u32x4* ta = stage;
  const u32x4* tb = stage + C::BK * C::CA;
  f32x16 sa[C::NMB], sb[C::NMB];
#pragma unroll
  for (int mb = 0; mb < C::NMB; ++mb) {
    const int r = 32 * mb + (lane & 31);
    f32x16 acc_a = zero16(), acc_b = zero16();
#pragma unroll
    for (int ks = 0; ks < DA / 16; ++ks) acc_a = mfma32(lds_row8<C::CA>(ta, r, 2 * ks + half), qa[ks], acc_a);
#pragma unroll
    for (int ks = 0; ks < DB / 16; ++ks) acc_b = mfma32(lds_row8<C::CB>(tb, r, 2 * ks + half), qb[ks], acc_b);
    sa[mb] = acc_a;
    sb[mb] = acc_b;
  }
  const int kbase = k0 + 4 * half;
  if (need_mask)
    fwd_tile_update<DA, DB, true>(st, sa, sb, ca, cb, kbase, NK, CAUSAL ? myq + off : NK);
  else
    fwd_tile_update<DA, DB, false>(st, sa, sb, ca, cb, kbase, NK, NK);
}

template <int DA, int DB, bool CAUSAL>
__global__ void __launch_bounds__(kThreads, (FwdCfg<DA, DB>::MINB))
kl_fwd_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
              const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
              int NQ, int NK, float ca, float cb,
              float* __restrict__ kl, float* __restrict__ lse_a, float* __restrict__ lse_b) {
  using C = FwdCfg<DA, DB>;
  // two statically distinct stages: the tile being read and the one being filled
  __shared__ u32x4 smem[2 * C::STAGE];

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

  if (ntiles > 0) dma.issue(rka, rkb, 0, smem, wave);
  wait_vmem();
  __syncthreads();
  for (int kt = 0; kt < ntiles; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < ntiles) dma.issue(rka, rkb, (kt + 1) * C::BK, smem + (buf ^ 1) * C::STAGE, wave);
    fwd_tile<DA, DB, CAUSAL>(smem + buf * C::STAGE, qa, qb, st, kt * C::BK, NK, qw, wlast, off, myq, ca, cb, lane);
    wait_vmem();
    __syncthreads();
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

}  // namespace streamkl
