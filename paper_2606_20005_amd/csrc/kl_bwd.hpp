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
// Where it can, a kernel folds |g| of a row into the row's exponent offsets
// (fold_row_stats), so that the exponentials are g P directly.
//
// MODE bit 0: produce the gradient of "b" (Setting 1); bit 1: of "a" (Setting 2).
#pragma once

#include "kl_common.hpp"

namespace streamkl {

// Activation of the attention scores: softmax (the paper's method) or the
// unnormalised sigmoid of Sec. 3.1 (see SigmoidRows in kl_fwd.hpp). With
// sigmoid scores A = sigmoid(S) the logit gradients of g L need no saved row
// statistic:  dS_b = g (A_b - A_a)(1 - A_b),
//             dS_a = g A_a (1 - A_a)(log A_a - log A_b).
constexpr int kActSoftmax = 0;
constexpr int kActSigmoid = 1;

template <int DA, int DB, int MODE>
struct BwdCfg {
  static constexpr int NW = 4;
  static constexpr int BR = 32 * NW;                     // resident rows per workgroup
  static constexpr int BS = 32;                          // streamed rows per tile
  static constexpr int CA = DA / 8, CB = DB / 8;
  static constexpr int STAGE = BS * (CA + CB);           // chunks per LDS stage
  static constexpr bool WANT_B = (MODE & 1) != 0;
  static constexpr bool WANT_A = (MODE & 2) != 0;
  // register estimate per lane: resident operands + two logit tiles + gradient
  // tiles + about 80 for operands in flight, addresses and row statistics;
  // two waves per SIMD leave 256.
  static constexpr int REGS = (DA + DB) / 4 + 32 + (WANT_A ? DA / 2 : 0) + (WANT_B ? DB / 2 : 0) + 80;
  // workgroups per CU; with four-wave workgroups also the waves per SIMD that
  // __launch_bounds__ takes as its second argument
  static constexpr int MINB = REGS <= 248 ? 2 : 1;
  static_assert(DA % 64 == 0 && DB % 64 == 0, "head dims must be multiples of 64");
  static_assert(MODE >= 1 && MODE <= 3, "at least one gradient");
};

// Row statistics in the form the inner loop uses.
struct RowStats {
  float lsa2, lsb2;  // LSE_a * log2 e, LSE_b * log2 e
  float g;           // upstream gradient of the row (0 for padding / empty rows)
  float dl;          // (LSE_a - LSE_b) + L
};

// Fold |g| into the exponent offsets of a row: g P_t = 2^(c_t raw - (LSE_t log2 e - log2 |g|)).
// A row with g = 0 gets +inf offsets (its P terms become 0). Subnormal |g|
// is scaled into the normal range first (the hardware log2 flushes
// subnormal inputs).
__device__ __forceinline__ RowStats fold_row_stats(RowStats s) {
  const float a = fabsf(s.g);
  const bool tiny = a < 0x1p-126f;
  const float l2g = __builtin_amdgcn_logf(tiny ? a * 0x1p64f : a) - (tiny ? 64.f : 0.f);   // -inf at 0
  s.lsa2 -= l2g;
  s.lsb2 -= l2g;
  return s;
}

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

// Saved values (LSE_a, LSE_b, L and, when given, g) of 64 consecutive query
// rows of one head, brought into LDS raw[4][64] by direct-to-LDS dword loads
// issued by one wave together with tile loads (rows past N_Q read as zeros;
// the dK kernel loads them one tile ahead). Once they have landed,
// stage_row_stats turns the 32 rows of a tile into the form the inner loop
// uses.
// (Sigmoid scores need g alone: ACT = kActSigmoid issues only that load, and
// the statistics pointers, which the caller may leave null, are not used.)
struct RowsDma {
  rsrc_t r_la, r_lb, r_kl, r_g;
  bool has_g;
  __device__ __forceinline__ RowsDma(const float* kl, const float* lse_a, const float* lse_b, const float* g,
                                     size_t head_row0, int NQ) {
    const uint32_t bytes = (uint32_t)NQ * 4u;
    has_g = g != nullptr;
    r_g = make_rsrc(has_g ? g + head_row0 : g, has_g ? bytes : 0u);
    r_la = make_rsrc(lse_a ? lse_a + head_row0 : lse_a, lse_a ? bytes : 0u);
    r_lb = make_rsrc(lse_b ? lse_b + head_row0 : lse_b, lse_b ? bytes : 0u);
    r_kl = make_rsrc(kl ? kl + head_row0 : kl, kl ? bytes : 0u);
  }
  template <int ACT>
  __device__ __forceinline__ void issue(int row0, float (*raw)[64], int lane) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t off = (uint32_t)(row0 + lane) * 4u;
    if constexpr (ACT == kActSoftmax) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r_la, (lds_void*)raw[0], 4, off, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r_lb, (lds_void*)raw[1], 4, off, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r_kl, (lds_void*)raw[2], 4, off, 0, 0, 0);
    }
    if (has_g) __builtin_amdgcn_raw_ptr_buffer_load_lds(r_g, (lds_void*)raw[3], 4, off, 0, 0, 0);
#endif
  }
};

// The statistics of one row of a streamed tile from its saved values (valid:
// the row exists), before the tile's fold decision; rows that do not exist
// or have no allowed key (LSE = -inf) contribute nothing.
__device__ __forceinline__ RowStats tile_row_stats(float la, float lb, float klv, float gv, bool valid) {
  RowStats s{0.f, 0.f, 0.f, 0.f};
  if (valid && la != kNegInf) {
    s.lsa2 = la * kLog2e;
    s.lsb2 = lb * kLog2e;
    s.g = gv;
    s.dl = (la - lb) + klv;
  }
  return s;
}
// ... and after it: a tile with no negative g folds |g| into the exponent
// offsets and stores g = 1, which keeps the unfolded path exact on it.
__device__ __forceinline__ RowStats finish_tile_row_stats(RowStats s, bool any_negative) {
  if (!any_negative) {
    s = fold_row_stats(s);
    s.g = 1.f;
  }
  return s;
}

// Statistics of a streamed 32-row tile in LDS: [lsa2, lsb2, g, dl][row], and
// in *fold whether g has been folded into lsa2, lsb2 (every g of the tile
// >= 0, the usual case; the stored g is then 1): the tile loop may then skip
// one multiply per distribution and element. Rows at tid >= BS idle.
template <int BS, int ACT = kActSoftmax>
__device__ __forceinline__ void stage_row_stats(const float (*raw)[64], int r0, int NQ, bool has_g,
                                                f32x4 (&dst)[4][BS / 4], int* fold, int tid) {
  if constexpr (ACT == kActSigmoid) {   // g alone, never folded
    if (tid < BS) {
      float* p = reinterpret_cast<float*>(&dst[0][0]);
      p[2 * BS + tid] = r0 + tid < NQ ? (has_g ? raw[3][tid] : 1.f) : 0.f;
      if (tid == 0) *fold = 0;
    }
    return;
  }
  RowStats s{0.f, 0.f, 0.f, 0.f};
  if (tid < BS)
    s = tile_row_stats(raw[0][tid], raw[1][tid], raw[2][tid], has_g ? raw[3][tid] : 1.f, r0 + tid < NQ);
  const bool any_negative = __builtin_amdgcn_ballot_w64(tid < BS && s.g < 0.f) != 0;
  if (tid < BS) {
    s = finish_tile_row_stats(s, any_negative);
    float* p = reinterpret_cast<float*>(&dst[0][0]);
    p[0 * BS + tid] = s.lsa2;
    p[1 * BS + tid] = s.lsb2;
    p[2 * BS + tid] = s.g;
    p[3 * BS + tid] = s.dl;
    if (tid == 0) *fold = any_negative ? 0 : 1;
  }
}

// ----------------------------------------------------------------------------
// Row statistics prepared ahead of the dK kernel. In the dK kernel the 32
// streamed rows of a tile lie along the registers of every lane, so their
// statistics pass through LDS; formed in the tile loop, one wave per tile
// does that work (stage_row_stats) while the other waves wait for it at the
// tile's barrier. kl_bwd_rowstats_kernel forms them for every tile of every
// head beforehand, with the same arithmetic bit for bit: tile T = head * ntq
// + t (ntq = ceil(N_Q / 32)) as stats[T][4][32] floats (lsa2, lsb2, g, dl by
// row) and fold[T], whether the tile's g are folded (the kernel is in
// kl_bwd_rowstats.hip). The dK kernel then streams each tile's 512 bytes and
// flag into LDS with its query tile.
// ----------------------------------------------------------------------------
constexpr int kRowStatsTile = 32;
constexpr int kRowStatsTilesPerBlock = 8;

// Direct-to-LDS loads of one prepared tile (512 bytes: two dword loads of the
// wave) and its fold flag (one lane), issued by one wave.
struct PreparedStatsDma {
  rsrc_t r_s, r_f;
  __device__ __forceinline__ PreparedStatsDma(const float* stats, const int* fold, size_t head_tile0, int ntq) {
    const bool on = stats != nullptr;
    r_s = make_rsrc(on ? stats + head_tile0 * 4 * kRowStatsTile : stats, on ? (uint32_t)ntq * 512u : 0u);
    r_f = make_rsrc(on ? fold + head_tile0 : fold, on ? (uint32_t)ntq * 4u : 0u);
  }
  __device__ __forceinline__ void issue(int t, float* dst, int* fold_dst, int lane) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t off = (uint32_t)t * 512u + (uint32_t)lane * 4u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r_s, (lds_void*)dst, 4, off, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r_s, (lds_void*)(dst + 64), 4, off + 256u, 0, 0, 0);
    if (lane == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(r_f, (lds_void*)fold_dst, 4, (uint32_t)t * 4u, 0, 0, 0);
#endif
  }
};

// Logit gradients of one element (raw dot products ra, rb). FOLD: the row's
// |g| is already folded into the exponent offsets (lsa2, lsb2 lowered by
// log2 |g|), so the exponentials are g P directly and the sign of g is
// applied elsewhere; otherwise g multiplies here.
template <bool WANT_A, bool WANT_B, bool FOLD = false, int ACT = kActSoftmax>
__device__ __forceinline__ void dlogits(float ra, float rb, bool ok, float ca, float cb, float sa, float sb,
                                        const RowStats& s, float& dsa, float& dsb) {
  if constexpr (ACT == kActSigmoid) {
    // ca, cb = s * log2(e): the helpers take the logits in base-2 units;
    // lr = log2 A_a - log2 A_b, needed for dS_a only
    if constexpr (WANT_A) {
      const SigmoidPair t = sigmoid_pair(ra * ca, rb * cb);
      if constexpr (WANT_B) dsb = ok ? s.g * ((t.b - t.a) * t.nb) : 0.f;
      dsa = ok ? s.g * (t.a * t.na) * (t.lr * kLn2) : 0.f;
    } else {
      const SigmoidTerms ta = sigmoid_terms(ra * ca), tb = sigmoid_terms(rb * cb);
      dsb = ok ? s.g * ((tb.a - ta.a) * tb.na) : 0.f;
    }
    return;
  }
  const float xa = ok ? __builtin_fmaf(ra, ca, -s.lsa2) : kNegInf;
  const float pa = exp2_fast(xa);
  if constexpr (WANT_B) {
    const float xb = ok ? __builtin_fmaf(rb, cb, -s.lsb2) : kNegInf;
    const float pb = exp2_fast(xb);
    dsb = FOLD ? pb - pa : s.g * (pb - pa);
  }
  if constexpr (WANT_A) {
    const float u = __builtin_fmaf(ra, sa, -__builtin_fmaf(rb, sb, s.dl));
    // p = 0 on a masked entry; select 0 rather than multiply, so that a
    // non-finite logit of a key the row may not see stays out of its row
    dsa = ok ? (FOLD ? pa * u : (s.g * pa) * u) : 0.f;
  }
}


// Wave priority around the matrix phases of a tile. Two waves share a SIMD:
// while one issues its MFMA chain at raised priority, the other's vector
// work fills the issue slots the chain leaves, which measured 3-4% faster
// for one gradient pair. With both pairs (twice the gradient MFMAs per
// tile) the raised priority starves the other wave's vector phase and
// measured 5% slower, so mode 3 keeps the default.
template <int MODE>
__device__ __forceinline__ void mfma_phase_begin() {
  if constexpr (MODE != 3) __builtin_amdgcn_s_setprio(1);
}
template <int MODE>
__device__ __forceinline__ void mfma_phase_end() {
  if constexpr (MODE != 3) __builtin_amdgcn_s_setprio(0);
}

// ----------------------------------------------------------------------------
// One streamed tile of one wave, shared by all backward kernels. The wave owns
// 32 resident rows (queries for dQ, keys for dK) held as MFMA B operands
// ra_op, rb_op; the stage holds 32 streamed rows of A and B. S = stage_rows x
// resident^T, so in the result lane l owns resident row l % 32 and 16 streamed
// rows (register i: streamed row 8 (i / 4) + 4 (l / 32) + i % 4). stats(i)
// returns the row statistics of element i and ok(i) whether element i is an
// allowed pair.
// ----------------------------------------------------------------------------
// ra_op(ks), rb_op(ks) return the resident operands of k-step ks (16 columns).
template <int DA, int DB, int MODE, bool MASK, bool FOLD, int ACT, typename OpA, typename OpB, typename StatsFn,
          typename OkFn>
__device__ __forceinline__ void bwd_dlogits_tile(const u32x4* stage, OpA ra_op, OpB rb_op, float ca, float cb,
                                                 float sa, float sb, int lane, StatsFn stats, OkFn ok,
                                                 float (&dsa)[16], float (&dsb)[16]) {
  using C = BwdCfg<DA, DB, MODE>;
  const int half = lane >> 5;
  const u32x4* ta = stage;
  const u32x4* tb = stage + C::BS * C::CA;
  const int r = lane & 31;
  f32x16 s_a = zero16(), s_b = zero16();
  mfma_phase_begin<MODE>();
#pragma unroll
  for (int ks = 0; ks < DA / 16; ++ks) s_a = mfma32(lds_row8<C::CA>(ta, r, 2 * ks + half), ra_op(ks), s_a);
#pragma unroll
  for (int ks = 0; ks < DB / 16; ++ks) s_b = mfma32(lds_row8<C::CB>(tb, r, 2 * ks + half), rb_op(ks), s_b);
  mfma_phase_end<MODE>();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const RowStats rs = stats(i);
    dlogits<C::WANT_A, C::WANT_B, FOLD, ACT>(s_a[i], s_b[i], MASK ? ok(i) : true, ca, cb, sa, sb, rs, dsa[i],
                                             dsb[i]);
  }
}

// Byte offsets within a stage of the transpose reads of the gradient
// contraction, for the calling lane: [32-column block nb][rows tr_row, tr_row
// + 8 of the first 16-row k-block]. The second k-block is 16 rows further,
// which the swizzle (a function of the row modulo 16) turns into a constant
// offset. They are computed once per kernel and passed through opaque(): the
// tile loops then address each stage as its array base plus these registers,
// with no per-tile address arithmetic, and the compiler still sees which
// stage array every read touches (it would otherwise wait for the loads in
// flight into the other stage before each read).
template <int DA, int DB, int MODE>
struct TrOffsets {
  using C = BwdCfg<DA, DB, MODE>;
  int a[C::WANT_A ? DA / 32 : 1][2];
  int b[C::WANT_B ? DB / 32 : 1][2];
  __device__ __forceinline__ explicit TrOffsets(int lane) {
    const int half = lane >> 5;
    // transpose-read addressing (see kl_common.hpp): row 4 * half + (lane % 16) / 4 of each
    // 16-row k-block, columns 16 * ((lane / 16) % 2) + 4 * (lane % 4) of each 32-column block.
    const int tr_row = 4 * half + ((lane & 15) >> 2);
    const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if constexpr (C::WANT_A) {
#pragma unroll
        for (int nb = 0; nb < DA / 32; ++nb) {
          const int e = 32 * nb + tr_col;
          a[nb][h] = opaque(chunk_slot<C::CA>(tr_row + 8 * h, e >> 3) * 16 + ((e >> 2) & 1) * 8);
        }
      }
      if constexpr (C::WANT_B) {
#pragma unroll
        for (int nb = 0; nb < DB / 32; ++nb) {
          const int e = 32 * nb + tr_col;
          b[nb][h] = opaque(C::BS * C::CA * 16 + chunk_slot<C::CB>(tr_row + 8 * h, e >> 3) * 16 + ((e >> 2) & 1) * 8);
        }
      }
    }
  }
};

// Gradient tiles of the resident rows from the logit gradients of one tile:
//   grad[resident][d] += sum_streamed dS[streamed][resident] * X[streamed][d]
// with X the streamed rows of the stage (transpose reads). dS, rounded to
// bf16, is the A operand as it lies in the registers.
template <int DA, int DB, int MODE>
__device__ __forceinline__ void bwd_grad_tile(const u32x4* stage, const float (&dsa)[16], const float (&dsb)[16],
                                              f32x16 (&ga)[(MODE & 2) ? DA / 32 : 1],
                                              f32x16 (&gb)[(MODE & 1) ? DB / 32 : 1],
                                              const TrOffsets<DA, DB, MODE>& to) {
  using C = BwdCfg<DA, DB, MODE>;
  mfma_phase_begin<MODE>();
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if constexpr (C::WANT_B) {
      const bf16x8 aop = pack8(dsb + 8 * s);
#pragma unroll
      for (int nb = 0; nb < DB / 32; ++nb) {
        const bf16x8 bop = cat8(lds_tr4_at(stage, to.b[nb][0] + 256 * C::CB * s),
                                lds_tr4_at(stage, to.b[nb][1] + 256 * C::CB * s));
        gb[nb] = mfma32(aop, bop, gb[nb]);
      }
    }
    if constexpr (C::WANT_A) {
      const bf16x8 aop = pack8(dsa + 8 * s);
#pragma unroll
      for (int nb = 0; nb < DA / 32; ++nb) {
        const bf16x8 bop = cat8(lds_tr4_at(stage, to.a[nb][0] + 256 * C::CA * s),
                                lds_tr4_at(stage, to.a[nb][1] + 256 * C::CA * s));
        ga[nb] = mfma32(aop, bop, ga[nb]);
      }
    }
  }
  mfma_phase_end<MODE>();
}

template <int DA, int DB, int MODE, bool MASK, bool FOLD, int ACT = kActSoftmax, typename StatsFn, typename OkFn>
__device__ __forceinline__ void bwd_tile(const u32x4* stage, const bf16x8 (&ra_op)[DA / 16],
                                         const bf16x8 (&rb_op)[DB / 16],
                                         f32x16 (&ga)[(MODE & 2) ? DA / 32 : 1],
                                         f32x16 (&gb)[(MODE & 1) ? DB / 32 : 1],
                                         float ca, float cb, float sa, float sb, int lane,
                                         StatsFn stats, OkFn ok, const TrOffsets<DA, DB, MODE>& to) {
  float dsa[16], dsb[16];
  bwd_dlogits_tile<DA, DB, MODE, MASK, FOLD, ACT>(stage, [&](int ks) { return ra_op[ks]; },
                                             [&](int ks) { return rb_op[ks]; }, ca, cb, sa, sb, lane, stats, ok,
                                             dsa, dsb);
  bwd_grad_tile<DA, DB, MODE>(stage, dsa, dsb, ga, gb, to);
}

// Resident rows of this lane as MFMA B operands (zero rows past n).
// dreal: the row length in global memory (D, or less for a padded head dim:
// the chunks past it are zeros).
template <int D>
__device__ __forceinline__ void load_resident(bf16x8 (&op)[D / 16], const uint16_t* X, size_t bh_rows, int row,
                                              int n, int half, int dreal = D) {
  const bool ok = row < n;
  const u32x4* p = reinterpret_cast<const u32x4*>(X + (bh_rows + (ok ? row : 0)) * dreal);
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const int c = 2 * ks + half;
    op[ks] = __builtin_bit_cast(bf16x8, ok && 8 * c < dreal ? p[c] : u32x4{0u, 0u, 0u, 0u});
  }
}

// Write one gradient tile: lane l, register i holds row base + 8 (i / 4) + 4 half + i % 4,
// column 32 nb + l % 32; the factor s of S = s Q K^T is applied here, times
// row_scale(i) when given. dreal: the row length in global memory (the
// 32-column blocks past it belong to a padded head dim and are dropped).
template <int D, typename RowScale>
__device__ __forceinline__ void write_grad(float* out, const f32x16 (&acc)[D / 32], size_t bh_rows, int base,
                                           int n, float s, int lane, int dreal, RowScale row_scale) {
  const int half = lane >> 5;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int row = base + 8 * (i >> 2) + 4 * half + (i & 3);
    if (row < n) {
      const float f = s * row_scale(i);
      float* o = out + (bh_rows + row) * dreal + (lane & 31);
#pragma unroll
      for (int nb = 0; nb < D / 32; ++nb)
        if (32 * nb < dreal) o[32 * nb] = acc[nb][i] * f;
    }
  }
}
template <int D>
__device__ __forceinline__ void write_grad(float* out, const f32x16 (&acc)[D / 32], size_t bh_rows, int base,
                                           int n, float s, int lane, int dreal = D) {
  write_grad<D>(out, acc, bh_rows, base, n, s, lane, dreal, [](int) { return 1.f; });
}

// ----------------------------------------------------------------------------
// dQ kernel: workgroup = 128 query rows of one (batch, head), streams key tiles.
// ----------------------------------------------------------------------------
template <int DA, int DB, bool CAUSAL, int MODE, int ACT = kActSoftmax, bool PD = false>
__global__ void __launch_bounds__(kThreads, (BwdCfg<DA, DB, MODE>::MINB))
kl_bwd_dq_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                 const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                 int NQ, int NK, int dra, int drb, float sa, float sb,
                 const float* __restrict__ kl, const float* __restrict__ lse_a,
                 const float* __restrict__ lse_b, const float* __restrict__ g,
                 float* __restrict__ dQa, float* __restrict__ dQb) {
  // PD: the head dims may be padded (the rows in memory are dra, drb long);
  // otherwise they are the compile-time ones and the runtime values unused
  if constexpr (!PD) {
    dra = DA;
    drb = DB;
  }
  using C = BwdCfg<DA, DB, MODE>;
  // Two stages of key tiles as two arrays, so that the compiler can tell
  // which stage each LDS read touches (the loop names each stage's array
  // explicitly, two tiles per trip).
  __shared__ u32x4 st0[C::STAGE];
  __shared__ u32x4 st1[C::STAGE];

  // the wave index is uniform: in a scalar register, so are the values derived from it
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), half = lane >> 5;
  const int TQ = (NQ + C::BR - 1) / C::BR;
  int bh, qt;
  head_block<CAUSAL, C::MINB>(TQ, bh, qt);
  if (CAUSAL) qt = TQ - 1 - qt;   // rank 0: the last rows, the longest
  const int q0 = qt * C::BR;
  const int off = NK - NQ;
  const int qw = q0 + 32 * wave;
  const int myq = qw + (lane & 31);
  const int wlast = min(qw + 31, NQ - 1);
  const float ca = sa * kLog2e, cb = sb * kLog2e;

  int ntiles = (NK + C::BS - 1) / C::BS;
  if (CAUSAL) {
    const int kmax = min(q0 + C::BR, NQ) - 1 + off;
    ntiles = kmax < 0 ? 0 : min(ntiles, kmax / C::BS + 1);
  }

  // |g| of the lane's row goes into its exponent offsets, its sign into the
  // written row
  // (sigmoid scores: only g, applied in the tile; kl and the LSEs are not read)
  constexpr bool FOLD = ACT == kActSoftmax;
  RowStats rs0{0.f, 0.f, 0.f, 0.f};
  if constexpr (ACT == kActSoftmax)
    rs0 = load_row_stats(kl, lse_a, lse_b, g, (size_t)bh * NQ + myq, myq < NQ);
  else if (myq < NQ)
    rs0.g = g ? g[(size_t)bh * NQ + myq] : 1.f;
  const float gsign = FOLD && rs0.g < 0.f ? -1.f : 1.f;
  const RowStats rs = FOLD ? fold_row_stats(rs0) : rs0;
  bf16x8 qa[DA / 16], qb[DB / 16];
  load_resident<DA>(qa, Qa, (size_t)bh * NQ, myq, NQ, half, dra);
  load_resident<DB>(qb, Qb, (size_t)bh * NQ, myq, NQ, half, drb);
  // complete before the tile loop: a wait for them inside the loop would
  // also wait for the loads of the next tile
  wait_vmem();

  f32x16 dqa[C::WANT_A ? DA / 32 : 1], dqb[C::WANT_B ? DB / 32 : 1];
#pragma unroll
  for (int n = 0; n < (C::WANT_A ? DA / 32 : 1); ++n) dqa[n] = zero16();
#pragma unroll
  for (int n = 0; n < (C::WANT_B ? DB / 32 : 1); ++n) dqb[n] = zero16();

  const rsrc_t rka = make_rsrc(Ka + (size_t)bh * NK * dra, (uint32_t)NK * dra * 2u);
  const rsrc_t rkb = make_rsrc(Kb + (size_t)bh * NK * drb, (uint32_t)NK * drb * 2u);
  const TileDma<C::BS, C::CA, C::CB> dma(tid, dra / 8, drb / 8);
  const int kmax_ok = CAUSAL ? myq + off : NK;

  const TrOffsets<DA, DB, MODE> tro(lane);
  auto tile = [&](const u32x4* stage, int kt) {
    const int k0 = kt * C::BS;
    bool active = qw < NQ;
    bool need_mask = k0 + C::BS > NK;
    if (CAUSAL) {
      active = active && (k0 <= wlast + off);
      need_mask = need_mask || (k0 + C::BS - 1 > qw + off);
    }
    if (!active) return;
    auto stats = [&](int) { return rs; };
    auto ok = [&](int i) {
      const int k = k0 + 8 * (i >> 2) + 4 * half + (i & 3);
      return k < NK && k <= kmax_ok;
    };
    if (opaque(need_mask))
      bwd_tile<DA, DB, MODE, true, FOLD, ACT>(stage, qa, qb, dqa, dqb, ca, cb, sa, sb, lane, stats, ok, tro);
    else
      bwd_tile<DA, DB, MODE, false, FOLD, ACT>(stage, qa, qb, dqa, dqb, ca, cb, sa, sb, lane, stats, ok, tro);
  };

  if (ntiles > 0) dma.issue(rka, rkb, 0, st0, wave, dra, drb);
  wait_vmem();
  __syncthreads();
  auto step = [&](const u32x4* cur, u32x4* nxt, int kt) {
    if (kt + 1 < ntiles) dma.issue(rka, rkb, (kt + 1) * C::BS, nxt, wave, dra, drb);
    tile(cur, kt);
    wait_vmem();
    __syncthreads();
  };
  for (int kt = 0; kt < ntiles; kt += 2) {
    step(st0, st1, kt);
    if (kt + 1 < ntiles) step(st1, st0, kt + 1);
  }

  // register i holds the row of lane 8 (i / 4) + 4 half + i % 4
  float rsign[16];
#pragma unroll
  for (int i = 0; i < 16; ++i)
    rsign[i] = __int_as_float(
        __builtin_amdgcn_ds_bpermute(4 * (8 * (i >> 2) + 4 * half + (i & 3)), __float_as_int(gsign)));
  auto row_sign = [&](int i) { return rsign[i]; };
  if constexpr (C::WANT_B) write_grad<DB>(dQb, dqb, (size_t)bh * NQ, qw, NQ, sb, lane, drb, row_sign);
  if constexpr (C::WANT_A) write_grad<DA>(dQa, dqa, (size_t)bh * NQ, qw, NQ, sa, lane, dra, row_sign);
}

// ----------------------------------------------------------------------------
// dK kernel: workgroup = 128 key rows of one (batch, head), streams query tiles
// together with their row statistics.
// ----------------------------------------------------------------------------
template <int DA, int DB, bool CAUSAL, int MODE, int ACT = kActSoftmax, bool PD = false>
__global__ void __launch_bounds__(kThreads, (BwdCfg<DA, DB, MODE>::MINB))
kl_bwd_dk_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                 const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                 int NQ, int NK, int dra, int drb, float sa, float sb,
                 const float* __restrict__ kl, const float* __restrict__ lse_a,
                 const float* __restrict__ lse_b, const float* __restrict__ g,
                 float* __restrict__ dKa, float* __restrict__ dKb,
                 const float* __restrict__ pstats, const int* __restrict__ pfold) {
  // PD: the head dims may be padded (the rows in memory are dra, drb long);
  // otherwise they are the compile-time ones and the runtime values unused
  if constexpr (!PD) {
    dra = DA;
    drb = DB;
  }
  using C = BwdCfg<DA, DB, MODE>;
  __shared__ u32x4 st0[C::STAGE];             // two stages of query tiles (two arrays: see the dQ kernel)
  __shared__ u32x4 st1[C::STAGE];
  __shared__ f32x4 sstat[2][4][C::BS / 4];    // their row statistics: [stage][lsa2, lsb2, g, dl][rows / 4]
  // saved row values as loaded, one tile ahead of the tiles (two arrays for
  // the same reason as the stages; tile t_begin + 2j uses the first)
  __shared__ float sraw0[4][64];
  __shared__ float sraw1[4][64];
  __shared__ int sfold[2];                    // per stage: g folded into the statistics

  // the wave index is uniform: in a scalar register, so are the values derived from it
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), half = lane >> 5;
  const int TK = (NK + C::BR - 1) / C::BR;
  int bh, kblk;
  head_block<CAUSAL, C::MINB>(TK, bh, kblk);   // causal rank 0: the first keys, seen by the most rows
  const int kb0 = kblk * C::BR;
  const int off = NK - NQ;
  const int kw = kb0 + 32 * wave;
  const int myk = kw + (lane & 31);
  const int wklast = min(kw + 31, NK - 1);
  const float ca = sa * kLog2e, cb = sb * kLog2e;

  const int ntq = (NQ + C::BS - 1) / C::BS;
  int t_begin = 0;
  if (CAUSAL) {
    const int qmin = kb0 - off;             // first row that sees key kb0
    t_begin = qmin <= 0 ? 0 : min(ntq, qmin / C::BS);
  }

  bf16x8 ka[DA / 16], kb[DB / 16];
  load_resident<DA>(ka, Ka, (size_t)bh * NK, myk, NK, half, dra);
  load_resident<DB>(kb, Kb, (size_t)bh * NK, myk, NK, half, drb);
  // complete before the tile loop: a wait for them inside the loop would
  // also wait for the loads of the next tile
  wait_vmem();

  f32x16 dka[C::WANT_A ? DA / 32 : 1], dkb[C::WANT_B ? DB / 32 : 1];
#pragma unroll
  for (int n = 0; n < (C::WANT_A ? DA / 32 : 1); ++n) dka[n] = zero16();
#pragma unroll
  for (int n = 0; n < (C::WANT_B ? DB / 32 : 1); ++n) dkb[n] = zero16();

  const rsrc_t rqa = make_rsrc(Qa + (size_t)bh * NQ * dra, (uint32_t)NQ * dra * 2u);
  const rsrc_t rqb = make_rsrc(Qb + (size_t)bh * NQ * drb, (uint32_t)NQ * drb * 2u);
  const TileDma<C::BS, C::CA, C::CB> dma(tid, dra / 8, drb / 8);

  const RowsDma rdma(kl, lse_a, lse_b, g, (size_t)bh * NQ, NQ);
  // prepared statistics (kl_bwd_rowstats_kernel), when the caller made them
  static_assert(C::BS == kRowStatsTile, "prepared statistics come in tiles of the streamed rows");
  const bool pre = ACT == kActSoftmax && pstats != nullptr;
  const PreparedStatsDma pdma(pre ? pstats : nullptr, pfold, (size_t)bh * ntq, ntq);

  const TrOffsets<DA, DB, MODE> tro(lane);
  auto tile = [&](const u32x4* stage, int buf, int t) {
    const f32x4 (&st)[4][C::BS / 4] = sstat[buf];
    const int r0 = t * C::BS;
    bool active = kw < NK;
    bool need_mask = r0 + C::BS > NQ;
    if (CAUSAL) {
      const int qlast = min(r0 + C::BS, NQ) - 1;
      active = active && (qlast + off >= kw);
      need_mask = need_mask || (wklast > r0 + off);
    }
    if (!active) return;
    // element i of this lane is streamed row r0 + 8 (i / 4) + 4 half + i % 4
    auto stats = [&](int i) {
      const int grp = 2 * (i >> 2) + half;
      return RowStats{st[0][grp][i & 3], st[1][grp][i & 3], st[2][grp][i & 3], st[3][grp][i & 3]};
    };
    auto ok = [&](int i) {
      const int q = r0 + 8 * (i >> 2) + 4 * half + (i & 3);
      return q < NQ && (!CAUSAL || myk <= q + off);
    };
    // the general path also takes the tiles whose g could not be folded
    // (a third variant would cost registers everywhere)
    if constexpr (ACT == kActSigmoid) {
      if (opaque(need_mask))
        bwd_tile<DA, DB, MODE, true, false, ACT>(stage, ka, kb, dka, dkb, ca, cb, sa, sb, lane, stats, ok, tro);
      else
        bwd_tile<DA, DB, MODE, false, false, ACT>(stage, ka, kb, dka, dkb, ca, cb, sa, sb, lane, stats, ok, tro);
    } else if (opaque(need_mask || !sfold[buf])) {
      bwd_tile<DA, DB, MODE, true, false>(stage, ka, kb, dka, dkb, ca, cb, sa, sb, lane, stats, ok, tro);
    } else {
      bwd_tile<DA, DB, MODE, false, true>(stage, ka, kb, dka, dkb, ca, cb, sa, sb, lane, stats, ok, tro);
    }
  };

  // Without prepared statistics, the row values of tile t + 1 are turned
  // into statistics by wave 0 early in step t, while the tile is computed:
  // they were loaded with the previous tile, so no wait sits between the
  // end-of-step wait and barrier. With them, wave 0 streams tile t + 1's
  // statistics and flag straight into their stage during step t.
  auto stats_in = [&](int t, float (*raw)[64], int buf) {
    if (wave == 0) stage_row_stats<C::BS, ACT>(raw, t * C::BS, NQ, rdma.has_g, sstat[buf], &sfold[buf], tid);
  };
  auto pre_in = [&](int t, int buf) {
    if (wave == 0) pdma.issue(t, reinterpret_cast<float*>(&sstat[buf][0][0]), &sfold[buf], lane);
  };
  if (t_begin < ntq) {
    dma.issue(rqa, rqb, t_begin * C::BS, st0, wave, dra, drb);
    if (pre) {
      pre_in(t_begin, 0);
    } else if (wave == 0) {
      rdma.issue<ACT>(t_begin * C::BS, sraw0, lane);
      if (t_begin + 1 < ntq) rdma.issue<ACT>((t_begin + 1) * C::BS, sraw1, lane);
    }
    wait_vmem();
    if (!pre) stats_in(t_begin, sraw0, 0);
  }
  __syncthreads();
  // rnext holds the row values of tile t + 1; rfree receives those of t + 2
  auto step = [&](const u32x4* cur, u32x4* nxt, float (*rnext)[64], float (*rfree)[64], int t, int buf) {
    if (t + 1 < ntq) dma.issue(rqa, rqb, (t + 1) * C::BS, nxt, wave, dra, drb);
    if (pre) {
      if (t + 1 < ntq) pre_in(t + 1, buf ^ 1);
    } else {
      if (wave == 0 && t + 2 < ntq) rdma.issue<ACT>((t + 2) * C::BS, rfree, lane);
      if (t + 1 < ntq) stats_in(t + 1, rnext, buf ^ 1);
    }
    tile(cur, buf, t);
    wait_vmem();
    __syncthreads();
  };
  for (int t = t_begin; t < ntq; t += 2) {
    step(st0, st1, sraw1, sraw0, t, 0);
    if (t + 1 < ntq) step(st1, st0, sraw0, sraw1, t + 1, 1);
  }

  if constexpr (C::WANT_B) write_grad<DB>(dKb, dkb, (size_t)bh * NK, kw, NK, sb, lane, drb);
  if constexpr (C::WANT_A) write_grad<DA>(dKa, dka, (size_t)bh * NK, kw, NK, sa, lane, dra);
}

}  // namespace streamkl
