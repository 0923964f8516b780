// Backward kernels of the fused attention-KL (Sec. 4: Algorithms 2 and 3 and
// the transposed dK tiling of Sec. 4.1.1), separate-kernel strategy of
// Sec. 4.2: a query-owned kernel writes dQ, a key-owned kernel writes dK, each
// tile of each output has exactly one owner, so there are no atomics and the
// result is bitwise reproducible.
//
// Both kernels recompute S_a, S_b on the MFMA and the probabilities from the
// saved log-sum-exps, P_t = 2^(raw * s_t * log2 e - LSE_t * log2 e), then
//   dS_b = g (P_b - P_a)                                    (eq:kl-case1)
//   dS_a = g P_a (s_a raw_a - s_b raw_b - (LSE_a - LSE_b) - L)
//        = g P_a (r - L)                                    (eq:kl-case2, eq:stable-r)
// where "a" is the distribution in the first KL slot and "b" the second
// (the host swaps (1) and (2) for KL(P2||P1)). The logit tile of the first
// contraction is laid out so that its fp32 accumulator, rounded to bf16,
// is directly the A operand of the second contraction (the 16-row k-blocks
// are a permutation of the 32 rows); the other operand of the second
// contraction, K (for dQ) or Q (for dK), is read from the same LDS tile with
// gfx950 transpose reads (ds_read_b64_tr_b16). The factor s_t of
// S_t = s_t Q_t K_t^T is applied once when the gradient tile is written.
//
// MODE bit 0: produce the gradient of "b" (Setting 1); bit 1: of "a" (Setting 2).
#pragma once

#include "kl_common.hpp"

namespace streamkl {

template <int DA, int DB, int MODE>
struct BwdCfg {
  static constexpr int NW = 4;
  static constexpr int BR = 32 * NW;                     // resident rows per workgroup
  static constexpr int BS = 32;                          // streamed rows per tile
  static constexpr int CA = DA / 8, CB = DB / 8;
  static constexpr int STAGE = BS * (CA + CB);           // chunks per LDS stage
  static constexpr int CHT = STAGE / kThreads;
  static constexpr int CHT_A = BS * CA / kThreads;
  static constexpr bool WANT_B = (MODE & 1) != 0;
  static constexpr bool WANT_A = (MODE & 2) != 0;
  // register estimate: resident operands + two logit tiles + gradient tiles
  static constexpr int REGS = (DA + DB) / 4 + 32 + (WANT_A ? DA / 2 : 0) + (WANT_B ? DB / 2 : 0) + CHT * 4;
  static constexpr int MINB = REGS <= 176 ? 2 : 1;
  static_assert(DA % 64 == 0 && DB % 64 == 0, "head dims must be multiples of 64");
  static_assert(STAGE % kThreads == 0 && (BS * CA) % kThreads == 0, "staging split");
  static_assert(MODE >= 1 && MODE <= 3, "at least one gradient");
};

// Row statistics in the form the inner loop uses.
struct RowStats {
  float lsa2, lsb2;  // LSE_a * log2 e, LSE_b * log2 e
  float g;           // upstream gradient of the row (0 for padding / empty rows)
  float dl;          // (LSE_a - LSE_b) + L
};

__device__ __forceinline__ RowStats load_row_stats(const float* kl, const float* lse_a, const float* lse_b,
                                                   const float* g, size_t ri, bool valid) {
  RowStats s{0.f, 0.f, 0.f, 0.f};
  if (valid) {
    const float la = lse_a[ri];
    if (la != kNegInf) {   // rows with no allowed key (LSE = -inf) contribute nothing
      const float lb = lse_b[ri];
      s.lsa2 = la * kLog2e;
      s.lsb2 = lb * kLog2e;
      s.g = g ? g[ri] : 1.f;
      s.dl = (la - lb) + kl[ri];
    }
  }
  return s;
}

// Logit gradients of one element (raw dot products ra, rb).
template <bool WANT_A, bool WANT_B>
__device__ __forceinline__ void dlogits(float ra, float rb, bool ok, float ca, float cb, float sa, float sb,
                                        const RowStats& s, float& dsa, float& dsb) {
  const float xa = ok ? __builtin_fmaf(ra, ca, -s.lsa2) : kNegInf;
  const float pa = exp2_fast(xa);
  if (WANT_B) {
    const float xb = ok ? __builtin_fmaf(rb, cb, -s.lsb2) : kNegInf;
    const float pb = exp2_fast(xb);
    dsb = s.g * (pb - pa);
  }
  if (WANT_A) {
    const float u = __builtin_fmaf(ra, sa, -__builtin_fmaf(rb, sb, s.dl));
    dsa = (s.g * pa) * u;
  }
}

// ----------------------------------------------------------------------------
// dQ kernel: workgroup = 128 query rows of one (batch, head), streams key tiles.
// ----------------------------------------------------------------------------
template <int DA, int DB, bool CAUSAL, int MODE>
__global__ void __launch_bounds__(kThreads, (BwdCfg<DA, DB, MODE>::MINB))
kl_bwd_dq_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                 const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                 int NQ, int NK, float sa, float sb,
                 const float* __restrict__ kl, const float* __restrict__ lse_a,
                 const float* __restrict__ lse_b, const float* __restrict__ g,
                 float* __restrict__ dQa, float* __restrict__ dQb) {
  using C = BwdCfg<DA, DB, MODE>;
  __shared__ uint4 smem[2 * C::STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int TQ = (NQ + C::BR - 1) / C::BR;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int bh = logical / TQ;
  int qt = logical - bh * TQ;
  if (CAUSAL) qt = TQ - 1 - qt;
  const int q0 = qt * C::BR;
  const int off = NK - NQ;
  const int qw = q0 + 32 * wave;
  const int myq = qw + (lane & 31);
  const float ca = sa * kLog2e, cb = sb * kLog2e;

  int ntiles = (NK + C::BS - 1) / C::BS;
  if (CAUSAL) {
    const int kmax = min(q0 + C::BR, NQ) - 1 + off;
    ntiles = kmax < 0 ? 0 : min(ntiles, kmax / C::BS + 1);
  }

  const RowStats rs = load_row_stats(kl, lse_a, lse_b, g, (size_t)bh * NQ + myq, myq < NQ);

  bf16x8 qa[DA / 16], qb[DB / 16];
  {
    const bool okq = myq < NQ;
    const uint4* pa = reinterpret_cast<const uint4*>(Qa + ((size_t)bh * NQ + (okq ? myq : 0)) * DA);
    const uint4* pb = reinterpret_cast<const uint4*>(Qb + ((size_t)bh * NQ + (okq ? myq : 0)) * DB);
#pragma unroll
    for (int ks = 0; ks < DA / 16; ++ks)
      qa[ks] = __builtin_bit_cast(bf16x8, okq ? pa[2 * ks + half] : make_uint4(0, 0, 0, 0));
#pragma unroll
    for (int ks = 0; ks < DB / 16; ++ks)
      qb[ks] = __builtin_bit_cast(bf16x8, okq ? pb[2 * ks + half] : make_uint4(0, 0, 0, 0));
  }

  f32x16 dqa[C::WANT_A ? DA / 32 : 1], dqb[C::WANT_B ? DB / 32 : 1];
#pragma unroll
  for (int n = 0; n < (C::WANT_A ? DA / 32 : 1); ++n) dqa[n] = zero16();
#pragma unroll
  for (int n = 0; n < (C::WANT_B ? DB / 32 : 1); ++n) dqb[n] = zero16();

  const uint4* gKa = reinterpret_cast<const uint4*>(Ka + (size_t)bh * NK * DA);
  const uint4* gKb = reinterpret_cast<const uint4*>(Kb + (size_t)bh * NK * DB);
  uint4 stg[C::CHT];
  auto gload = [&](int kt) {
    const int k0 = kt * C::BS;
#pragma unroll
    for (int i = 0; i < C::CHT; ++i) {
      const int p = tid + kThreads * i;
      if (i < C::CHT_A) {
        const int r = p / C::CA, c = p - r * C::CA;
        stg[i] = gKa[(size_t)min(k0 + r, NK - 1) * C::CA + c];
      } else {
        const int pp = p - C::BS * C::CA;
        const int r = pp / C::CB, c = pp - r * C::CB;
        stg[i] = gKb[(size_t)min(k0 + r, NK - 1) * C::CB + c];
      }
    }
  };
  auto lstore = [&](int buf) {
    uint4* base = smem + buf * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::CHT; ++i) {
      const int p = tid + kThreads * i;
      if (i < C::CHT_A) {
        const int r = p / C::CA, c = p - r * C::CA;
        base[chunk_slot<C::CA>(r, c)] = stg[i];
      } else {
        const int pp = p - C::BS * C::CA;
        const int r = pp / C::CB, c = pp - r * C::CB;
        base[C::BS * C::CA + chunk_slot<C::CB>(r, c)] = stg[i];
      }
    }
  };

  const int wlast = min(qw + 31, NQ - 1);
  // transpose-read addressing of this lane (see kl_common.hpp): row 4 * half + lane/4 % 4
  // of each 16-row k-block, columns 16 * (lane/16 % 2) + 4 * (lane % 4) of each 32-column block.
  const int tr_row = 4 * half + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  if (ntiles > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int kt = 0; kt < ntiles; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < ntiles) gload(kt + 1);
    const int k0 = kt * C::BS;
    bool active = qw < NQ;
    bool need_mask = k0 + C::BS > NK;
    if (CAUSAL) {
      active = active && (k0 <= wlast + off);
      need_mask = need_mask || (k0 + C::BS - 1 > qw + off);
    }
    if (active) {
      const uint4* ta = smem + buf * C::STAGE;
      const uint4* tb = ta + C::BS * C::CA;
      const int r = lane & 31;
      f32x16 s_a = zero16(), s_b = zero16();
#pragma unroll
      for (int ks = 0; ks < DA / 16; ++ks) s_a = mfma32(lds_row8<C::CA>(ta, r, 2 * ks + half), qa[ks], s_a);
#pragma unroll
      for (int ks = 0; ks < DB / 16; ++ks) s_b = mfma32(lds_row8<C::CB>(tb, r, 2 * ks + half), qb[ks], s_b);
      float dsa[16], dsb[16];
      const int kmax_ok = CAUSAL ? myq + off : NK;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int k = k0 + 8 * (i >> 2) + 4 * half + (i & 3);
        const bool ok = need_mask ? (k < NK && k <= kmax_ok) : true;
        dlogits<C::WANT_A, C::WANT_B>(s_a[i], s_b[i], ok, ca, cb, sa, sb, rs, dsa[i], dsb[i]);
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        if (C::WANT_B) {
          const bf16x8 aop = pack8(dsb + 8 * s);
#pragma unroll
          for (int nb = 0; nb < DB / 32; ++nb) {
            const bf16x8 bop = cat8(lds_tr4<C::CB>(tb, 16 * s + tr_row, 32 * nb + tr_col),
                                    lds_tr4<C::CB>(tb, 16 * s + 8 + tr_row, 32 * nb + tr_col));
            dqb[nb] = mfma32(aop, bop, dqb[nb]);
          }
        }
        if (C::WANT_A) {
          const bf16x8 aop = pack8(dsa + 8 * s);
#pragma unroll
          for (int nb = 0; nb < DA / 32; ++nb) {
            const bf16x8 bop = cat8(lds_tr4<C::CA>(ta, 16 * s + tr_row, 32 * nb + tr_col),
                                    lds_tr4<C::CA>(ta, 16 * s + 8 + tr_row, 32 * nb + tr_col));
            dqa[nb] = mfma32(aop, bop, dqa[nb]);
          }
        }
      }
    }
    if (kt + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
  }

  // Write: lane l, register i holds row qw + 8 (i / 4) + 4 half + i % 4, column 32 nb + l % 32.
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int q = qw + 8 * (i >> 2) + 4 * half + (i & 3);
    if (q < NQ) {
      if (C::WANT_B) {
        float* out = dQb + ((size_t)bh * NQ + q) * DB + (lane & 31);
#pragma unroll
        for (int nb = 0; nb < DB / 32; ++nb) out[32 * nb] = dqb[nb][i] * sb;
      }
      if (C::WANT_A) {
        float* out = dQa + ((size_t)bh * NQ + q) * DA + (lane & 31);
#pragma unroll
        for (int nb = 0; nb < DA / 32; ++nb) out[32 * nb] = dqa[nb][i] * sa;
      }
    }
  }
}

// ----------------------------------------------------------------------------
// dK kernel: workgroup = 128 key rows of one (batch, head), streams query tiles
// together with their row statistics.
// ----------------------------------------------------------------------------
template <int DA, int DB, bool CAUSAL, int MODE>
__global__ void __launch_bounds__(kThreads, (BwdCfg<DA, DB, MODE>::MINB))
kl_bwd_dk_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                 const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                 int NQ, int NK, float sa, float sb,
                 const float* __restrict__ kl, const float* __restrict__ lse_a,
                 const float* __restrict__ lse_b, const float* __restrict__ g,
                 float* __restrict__ dKa, float* __restrict__ dKb) {
  using C = BwdCfg<DA, DB, MODE>;
  __shared__ uint4 smem[2 * C::STAGE];
  __shared__ f32x4 sstat[2][4][C::BS / 4];   // [stage][lsa2, lsb2, g, dl][4 rows]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int TK = (NK + C::BR - 1) / C::BR;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int bh = logical / TK;
  const int kt_blk = logical - bh * TK;     // causal: low key tiles see the most rows, so they go first
  const int kb0 = kt_blk * C::BR;
  const int off = NK - NQ;
  const int kw = kb0 + 32 * wave;           // first key of this wave
  const int myk = kw + (lane & 31);
  const float ca = sa * kLog2e, cb = sb * kLog2e;

  const int ntq = (NQ + C::BS - 1) / C::BS;
  int t_begin = 0;
  if (CAUSAL) {
    const int qmin = kb0 - off;             // first row that sees key kb0
    t_begin = qmin <= 0 ? 0 : min(ntq, qmin / C::BS);
  }

  // K rows of this lane as MFMA B operands.
  bf16x8 ka[DA / 16], kb[DB / 16];
  {
    const bool okk = myk < NK;
    const uint4* pa = reinterpret_cast<const uint4*>(Ka + ((size_t)bh * NK + (okk ? myk : 0)) * DA);
    const uint4* pb = reinterpret_cast<const uint4*>(Kb + ((size_t)bh * NK + (okk ? myk : 0)) * DB);
#pragma unroll
    for (int ks = 0; ks < DA / 16; ++ks)
      ka[ks] = __builtin_bit_cast(bf16x8, okk ? pa[2 * ks + half] : make_uint4(0, 0, 0, 0));
#pragma unroll
    for (int ks = 0; ks < DB / 16; ++ks)
      kb[ks] = __builtin_bit_cast(bf16x8, okk ? pb[2 * ks + half] : make_uint4(0, 0, 0, 0));
  }

  f32x16 dka[C::WANT_A ? DA / 32 : 1], dkb[C::WANT_B ? DB / 32 : 1];
#pragma unroll
  for (int n = 0; n < (C::WANT_A ? DA / 32 : 1); ++n) dka[n] = zero16();
#pragma unroll
  for (int n = 0; n < (C::WANT_B ? DB / 32 : 1); ++n) dkb[n] = zero16();

  const uint4* gQa = reinterpret_cast<const uint4*>(Qa + (size_t)bh * NQ * DA);
  const uint4* gQb = reinterpret_cast<const uint4*>(Qb + (size_t)bh * NQ * DB);
  uint4 stg[C::CHT];
  RowStats sst{0.f, 0.f, 0.f, 0.f};
  auto gload = [&](int t) {
    const int r0 = t * C::BS;
#pragma unroll
    for (int i = 0; i < C::CHT; ++i) {
      const int p = tid + kThreads * i;
      if (i < C::CHT_A) {
        const int r = p / C::CA, c = p - r * C::CA;
        stg[i] = gQa[(size_t)min(r0 + r, NQ - 1) * C::CA + c];
      } else {
        const int pp = p - C::BS * C::CA;
        const int r = pp / C::CB, c = pp - r * C::CB;
        stg[i] = gQb[(size_t)min(r0 + r, NQ - 1) * C::CB + c];
      }
    }
    if (tid < C::BS) {
      const int q = r0 + tid;
      sst = load_row_stats(kl, lse_a, lse_b, g, (size_t)bh * NQ + q, q < NQ);
    }
  };
  auto lstore = [&](int buf) {
    uint4* base = smem + buf * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::CHT; ++i) {
      const int p = tid + kThreads * i;
      if (i < C::CHT_A) {
        const int r = p / C::CA, c = p - r * C::CA;
        base[chunk_slot<C::CA>(r, c)] = stg[i];
      } else {
        const int pp = p - C::BS * C::CA;
        const int r = pp / C::CB, c = pp - r * C::CB;
        base[C::BS * C::CA + chunk_slot<C::CB>(r, c)] = stg[i];
      }
    }
    if (tid < C::BS) {
      float* s = reinterpret_cast<float*>(&sstat[buf][0][0]);
      s[0 * C::BS + tid] = sst.lsa2;
      s[1 * C::BS + tid] = sst.lsb2;
      s[2 * C::BS + tid] = sst.g;
      s[3 * C::BS + tid] = sst.dl;
    }
  };

  const int wklast = min(kw + 31, NK - 1);
  const int tr_row = 4 * half + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  if (t_begin < ntq) {
    gload(t_begin);
    lstore(0);
  }
  __syncthreads();
  for (int t = t_begin; t < ntq; ++t) {
    const int buf = (t - t_begin) & 1;
    if (t + 1 < ntq) gload(t + 1);
    const int r0 = t * C::BS;
    bool active = kw < NK;
    bool need_mask = r0 + C::BS > NQ;
    if (CAUSAL) {
      const int qlast = min(r0 + C::BS, NQ) - 1;
      active = active && (qlast + off >= kw);
      need_mask = need_mask || (wklast > r0 + off);
    }
    if (active) {
      const uint4* ta = smem + buf * C::STAGE;
      const uint4* tb = ta + C::BS * C::CA;
      const int r = lane & 31;
      f32x16 s_a = zero16(), s_b = zero16();
      // S[row][key]: A = Q rows from LDS, B = this wave's K rows.
#pragma unroll
      for (int ks = 0; ks < DA / 16; ++ks) s_a = mfma32(lds_row8<C::CA>(ta, r, 2 * ks + half), ka[ks], s_a);
#pragma unroll
      for (int ks = 0; ks < DB / 16; ++ks) s_b = mfma32(lds_row8<C::CB>(tb, r, 2 * ks + half), kb[ks], s_b);
      float dsa[16], dsb[16];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // rows 8 j + 4 half + 0..3 of the tile: one 16-byte read per statistic
        const int rr = 8 * j + 4 * half;
        const f32x4 vlsa = sstat[buf][0][rr / 4];
        const f32x4 vlsb = sstat[buf][1][rr / 4];
        const f32x4 vg = sstat[buf][2][rr / 4];
        const f32x4 vdl = sstat[buf][3][rr / 4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * j + e;
          const int q = r0 + rr + e;
          const bool ok = need_mask ? (q < NQ && (!CAUSAL || myk <= q + off)) : true;
          const RowStats rsq{vlsa[e], vlsb[e], vg[e], vdl[e]};
          dlogits<C::WANT_A, C::WANT_B>(s_a[i], s_b[i], ok, ca, cb, sa, sb, rsq, dsa[i], dsb[i]);
        }
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        if (C::WANT_B) {
          const bf16x8 aop = pack8(dsb + 8 * s);
#pragma unroll
          for (int nb = 0; nb < DB / 32; ++nb) {
            const bf16x8 bop = cat8(lds_tr4<C::CB>(tb, 16 * s + tr_row, 32 * nb + tr_col),
                                    lds_tr4<C::CB>(tb, 16 * s + 8 + tr_row, 32 * nb + tr_col));
            dkb[nb] = mfma32(aop, bop, dkb[nb]);
          }
        }
        if (C::WANT_A) {
          const bf16x8 aop = pack8(dsa + 8 * s);
#pragma unroll
          for (int nb = 0; nb < DA / 32; ++nb) {
            const bf16x8 bop = cat8(lds_tr4<C::CA>(ta, 16 * s + tr_row, 32 * nb + tr_col),
                                    lds_tr4<C::CA>(ta, 16 * s + 8 + tr_row, 32 * nb + tr_col));
            dka[nb] = mfma32(aop, bop, dka[nb]);
          }
        }
      }
    }
    if (t + 1 < ntq) lstore(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int k = kw + 8 * (i >> 2) + 4 * half + (i & 3);
    if (k < NK) {
      if (C::WANT_B) {
        float* out = dKb + ((size_t)bh * NK + k) * DB + (lane & 31);
#pragma unroll
        for (int nb = 0; nb < DB / 32; ++nb) out[32 * nb] = dkb[nb][i] * sb;
      }
      if (C::WANT_A) {
        float* out = dKa + ((size_t)bh * NK + k) * DA + (lane & 31);
#pragma unroll
        for (int nb = 0; nb < DA / 32; ++nb) out[32 * nb] = dka[nb][i] * sa;
      }
    }
  }
}

}  // namespace streamkl
