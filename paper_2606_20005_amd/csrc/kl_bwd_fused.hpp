// Fused backward kernel of the attention KL (Sec. 4.2, "Fused Backward
// Kernel"): one kernel visits every (query tile, key block) pair once and
// produces dK and dQ together.
//
// The grid is partitioned on the keys, as in the paper: a workgroup of four
// waves owns 128 keys of one (batch, head), each wave 32 of them as MFMA
// operands, and streams the query tiles (32 rows each, with their row
// statistics) through the two-stage LDS ring of the separate dK kernel. Per
// tile each wave recomputes S_a, S_b and the logit gradients exactly as the
// separate kernels do and accumulates its dK rows in registers (exclusive
// ownership, no atomics). The dQ rows of the tile receive contributions from
// every key block of the head, so they are added into dQ with fp32 atomics:
//
//   1. each wave stores its dS tile (32 keys x 32 query rows, bf16, the value
//      the second contraction consumes in the separate kernels too) into one
//      shared 128 x 32 LDS tile;
//   2. after a barrier the workgroup computes dQ_tile = dS^T-tile . K_block
//      over all 128 keys, the waves splitting the columns of dQ in 32-wide
//      blocks, with dS read back by transpose reads and K from an LDS copy of
//      the key block;
//   3. each output element of the 32 x d tile gets one atomic add per key
//      block.
//
// MODE selects the distributions as in the separate kernels; within a side
// a NULL dQ or dK pointer skips that output (the host passes NULL for a
// gradient nobody asked for).
//
// dQ must be zero on entry (the host launches a fill kernel first). The sum
// order of the atomics is not fixed, so dQ can differ from run to run in the
// last bits; dK is written by its owner and stays reproducible.
//
// dS LDS tile layout: row k (key of the block, 0..127) holds 32 query rows as
// eight 8-byte units of four bf16; unit u of row k sits at byte
// 64 k + 8 (u ^ (k / 4 mod 8)). The writes (each lane one key row, one unit
// per instruction) and the transpose reads (four consecutive key rows, eight
// consecutive units per 32 lanes) both touch 64 distinct banks.
#pragma once

#include "kl_bwd.hpp"

namespace streamkl {

template <int DA, int DB, int MODE>
struct FusedCfg {
  using Base = BwdCfg<DA, DB, MODE>;
  static constexpr int BR = Base::BR;                      // keys per workgroup
  static constexpr int BS = Base::BS;                      // query rows per streamed tile
  static constexpr int CA = Base::CA, CB = Base::CB;
  static constexpr bool WANT_A = Base::WANT_A, WANT_B = Base::WANT_B;
  static constexpr int NCB_A = WANT_A ? DA / 32 : 0;       // 32-column blocks of dQ_a
  static constexpr int NCB_B = WANT_B ? DB / 32 : 0;
  static constexpr int ITEMS = NCB_A + NCB_B;              // dQ column blocks shared by the waves
  // LDS, in 16-byte chunks
  static constexpr int RING = 2 * Base::STAGE;
  static constexpr int KRES_A = WANT_A ? BR * CA : 0;      // key block copies for the dQ contraction
  static constexpr int KRES_B = WANT_B ? BR * CB : 0;
  static constexpr int DS_CH = BR * BS * 2 / 16;           // one dS tile (bf16)
  static constexpr int NDS = (WANT_A ? 1 : 0) + (WANT_B ? 1 : 0);
  static constexpr int CHUNKS = RING + KRES_A + KRES_B + NDS * DS_CH;
  static constexpr int LDS_BYTES = 16 * CHUNKS + 2 * 4 * BS * 4 + 2 * 4 * 64 * 4 + 16;
  static constexpr int LDS_LIMIT = 160 * 1024;
  static constexpr bool FITS = LDS_BYTES <= LDS_LIMIT;
  static constexpr int MINB = (Base::MINB == 2 && 2 * LDS_BYTES <= LDS_LIMIT) ? 2 : 1;
};

// Byte offset of unit u (query rows 4u .. 4u + 3) of key row k in a dS tile.
__device__ __forceinline__ int ds_unit_byte(int k, int u) { return 64 * k + 8 * (u ^ ((k >> 2) & 7)); }

// Store this lane's 16 logit gradients (key row k; register i holds query row
// 8 (i / 4) + 4 half + i % 4) as bf16 into a dS tile.
__device__ __forceinline__ void store_ds(u32x4* tile, int k, int half, const float (&ds)[16]) {
  char* base = reinterpret_cast<char*>(tile);
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    bf16x4 v;
#pragma unroll
    for (int t = 0; t < 4; ++t) v[t] = (__bf16)ds[4 * b + t];
    *reinterpret_cast<bf16x4*>(base + ds_unit_byte(k, 2 * b + half)) = v;
  }
}

// Per-lane byte offsets of the transpose reads of the dQ contraction for
// 32-column block cb (see dq_block_mma), computed once per kernel and passed
// through opaque() for the reason given at TrOffsets.
//
// A operand (dS, query row lane % 32): two transpose reads of four key rows
// each, keys 16 j + 8 half + 4 rho + 0..3, unit u = 4 g + lane % 4. In the dS
// layout the unit swizzle of those rows is (4 (j % 2) + 2 half + rho), so the
// byte address is a per-lane base for each (rho, j % 2) plus 1024 j.
// B operand (K, column 32 cb + lane % 32): the same key rows of the key block
// copy; its swizzle depends only on the row modulo 16, so the address is a
// per-lane base per rho plus 16 j rows. All group offsets are immediates.
struct DqOffsets {
  int a[2][2];   // [rho][j % 2]
  int b[2];      // [rho]
};

template <int CPR>
__device__ __forceinline__ DqOffsets dq_offsets(int lane, int cb) {
  DqOffsets o;
  const int half = lane >> 5, g = (lane >> 4) & 1, jj = lane & 15;
  const int u = 4 * g + (jj & 3);
  const int col = 32 * cb + 16 * g + 4 * (jj & 3);
#pragma unroll
  for (int rho = 0; rho < 2; ++rho) {
    const int kr = 8 * half + 4 * rho + (jj >> 2);   // key row of group 0
#pragma unroll
    for (int par = 0; par < 2; ++par) o.a[rho][par] = opaque(ds_unit_byte(kr + 16 * par, u) - 1024 * par);
    o.b[rho] = opaque(chunk_slot<CPR>(kr, col >> 3) * 16 + ((col >> 2) & 1) * 8);
  }
  return o;
}

// dQ contribution of one 32-column block: sum over the key block's 16-key
// groups j < jend (of NJ) of dS[q][keys] . K[keys][32 cb ..].
template <int CPR, int NJ>
__device__ __forceinline__ f32x16 dq_block_mma(const u32x4* ds_tile, const u32x4* kres, const DqOffsets& o,
                                               int jend) {
  f32x16 acc = zero16();
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (j < jend) {
      const bf16x8 aop = cat8(lds_tr4_at(ds_tile, o.a[0][j & 1] + 1024 * j), lds_tr4_at(ds_tile, o.a[1][j & 1] + 1024 * j));
      const bf16x8 bop = cat8(lds_tr4_at(kres, o.b[0] + 256 * CPR * j), lds_tr4_at(kres, o.b[1] + 256 * CPR * j));
      acc = mfma32(aop, bop, acc);
    }
  }
  return acc;
}

// One atomic add per element of the 32 x 32 dQ tile (kDqAtomicsPerBlock per
// lane). When every row of the tile exists and sees the key block (FULL),
// all of them are issued unconditionally, in straight-line code, so the
// number of vector memory instructions is known (the end-of-tile wait relies
// on it); otherwise lanes without a row are masked off.
constexpr int kDqAtomicsPerBlock = 16;
static_assert(sizeof(f32x16) / sizeof(float) == kDqAtomicsPerBlock, "one atomic per accumulator register");
template <int D, bool CAUSAL, bool FULL>
__device__ __forceinline__ void dq_block_add(const f32x16& acc, int cb, int lane, float* __restrict__ dq,
                                             size_t row_base, int q0, int NQ, int qmin_seen, float s) {
  const int half = lane >> 5;
  const int qh = q0 + 4 * half;   // row of register 0; register i adds 8 (i / 4) + i % 4
  float* out = dq + (row_base + qh) * D + 32 * cb + (lane & 31);
#pragma unroll
  for (int i = 0; i < kDqAtomicsPerBlock; ++i) {
    const int ri = 8 * (i >> 2) + (i & 3);
    const int q = qh + ri;
    if (FULL || (q < NQ && (!CAUSAL || q >= qmin_seen))) atomic_add_global(out + ri * D, acc[i] * s);
  }
}

template <int DA, int DB, bool CAUSAL, int MODE>
__global__ void __launch_bounds__(kThreads, (FusedCfg<DA, DB, MODE>::MINB))
kl_bwd_fused_kernel(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Ka,
                    const uint16_t* __restrict__ Qb, const uint16_t* __restrict__ Kb,
                    int NQ, int NK, float sa, float sb,
                    const float* __restrict__ kl, const float* __restrict__ lse_a,
                    const float* __restrict__ lse_b, const float* __restrict__ g,
                    float* __restrict__ dQa, float* __restrict__ dQb,
                    float* __restrict__ dKa, float* __restrict__ dKb) {
  using C = FusedCfg<DA, DB, MODE>;
  using BC = typename C::Base;
  static_assert(C::FITS, "fused backward does not fit in LDS for these head dims");
  // Separate arrays for every LDS region: the compiler can then tell that the
  // reads of one region never alias the direct-to-LDS loads landing in
  // another, and inserts no waits for those loads (the tile loop names each
  // stage's array explicitly, two tiles per trip).
  // Each stage holds a query tile and, after it, the saved values of its rows
  // as loaded (4 x 64 floats): all direct-to-LDS loads of the loop then
  // target the two stage arrays only, which keeps the compiler's tracking of
  // those loads exact.
  constexpr int RAW = 64;                                           // chunks of raw row values
  __shared__ u32x4 st0[BC::STAGE + RAW];                            // query tile + raw row values, stage 0
  __shared__ u32x4 st1[BC::STAGE + RAW];                            // stage 1
  __shared__ u32x4 kres_a[C::WANT_A ? C::BR * C::CA : 1];           // key block copies
  __shared__ u32x4 kres_b[C::WANT_B ? C::BR * C::CB : 1];
  __shared__ u32x4 ds_a[C::WANT_A ? C::DS_CH : 1];                  // dS tiles
  __shared__ u32x4 ds_b[C::WANT_B ? C::DS_CH : 1];
  __shared__ f32x4 sstat[2][4][C::BS / 4];                          // row statistics of the stages
  __shared__ int sfold[2];                                          // per stage: g folded into them
  auto raw_of = [](const u32x4* stage) { return reinterpret_cast<const float (*)[64]>(stage + BC::STAGE); };

  // the wave index is uniform: in a scalar register, so are the values derived from it
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), half = lane >> 5;
  const int TK = (NK + C::BR - 1) / C::BR;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int bh = logical / TK;
  const int kb0 = (logical - bh * TK) * C::BR;
  const int off = NK - NQ;
  const int kw = kb0 + 32 * wave;
  const int kloc = 32 * wave + (lane & 31);   // key row within the block
  const int myk = kb0 + kloc;
  const int wklast = min(kw + 31, NK - 1);
  const int blast = min(kb0 + C::BR, NK) - 1;
  const float ca = sa * kLog2e, cb = sb * kLog2e;

  const int ntq = (NQ + C::BS - 1) / C::BS;
  int t_begin = 0;
  if (CAUSAL) {
    const int qmin = kb0 - off;   // first row that sees key kb0
    t_begin = qmin <= 0 ? 0 : min(ntq, qmin / C::BS);
  }

  // The logit operands of a side whose key block is copied to LDS are read
  // from there; the other side's stay in registers.
  bf16x8 ka[C::WANT_A ? 1 : DA / 16], kb[C::WANT_B ? 1 : DB / 16];
  if constexpr (!C::WANT_A) load_resident<DA>(ka, Ka, (size_t)bh * NK, myk, NK, half);
  if constexpr (!C::WANT_B) load_resident<DB>(kb, Kb, (size_t)bh * NK, myk, NK, half);
  wait_vmem();   // before the tile loop, whose first use would otherwise wait in every trip
  // kres_row is made opaque once per tile so that the compiler cannot hoist
  // these loop-invariant reads out of the tile loop (into registers).
  int kres_row = kloc;
  auto op_a = [&](int ks) {
    if constexpr (C::WANT_A) return lds_row8<C::CA>(kres_a, kres_row, 2 * ks + half);
    else return ka[ks];
  };
  auto op_b = [&](int ks) {
    if constexpr (C::WANT_B) return lds_row8<C::CB>(kres_b, kres_row, 2 * ks + half);
    else return kb[ks];
  };

  f32x16 dka[C::WANT_A ? DA / 32 : 1], dkb[C::WANT_B ? DB / 32 : 1];
#pragma unroll
  for (int n = 0; n < (C::WANT_A ? DA / 32 : 1); ++n) dka[n] = zero16();
#pragma unroll
  for (int n = 0; n < (C::WANT_B ? DB / 32 : 1); ++n) dkb[n] = zero16();

  const rsrc_t rqa = make_rsrc(Qa + (size_t)bh * NQ * DA, (uint32_t)NQ * DA * 2u);
  const rsrc_t rqb = make_rsrc(Qb + (size_t)bh * NQ * DB, (uint32_t)NQ * DB * 2u);
  const TileDma<C::BS, C::CA, C::CB> dma(tid);
  const RowsDma rdma(kl, lse_a, lse_b, g, (size_t)bh * NQ, NQ);

  // key block copies (rows past N_K read as zeros)
  if constexpr (C::WANT_A) {
    const rsrc_t rka = make_rsrc(Ka + (size_t)bh * NK * DA, (uint32_t)NK * DA * 2u);
    const TileDma<C::BR, C::CA, 0> kdma(tid);
    kdma.issue(rka, rka, kb0, kres_a, wave);
  }
  if constexpr (C::WANT_B) {
    const rsrc_t rkb = make_rsrc(Kb + (size_t)bh * NK * DB, (uint32_t)NK * DB * 2u);
    const TileDma<C::BR, C::CB, 0> kdma(tid);
    kdma.issue(rkb, rkb, kb0, kres_b, wave);
  }

  // Every key block of a head adds into the same dQ tiles. Each block visits
  // its query tiles in a rotated order, starting at its own index, so that the
  // blocks running at the same time add into different dQ tiles.
  const int nt = ntq - t_begin;
  const int rot = nt > 0 ? (kb0 / C::BR) % nt : 0;
  auto tile_at = [&](int i) {
    const int k = i + rot;
    return t_begin + (k < nt ? k : k - nt);
  };
  const TrOffsets<DA, DB, MODE> tro(lane);
  auto stage_in = [&](int t, u32x4* dst) {
    dma.issue(rqa, rqb, t * C::BS, dst, wave);
    if (wave == 0) rdma.issue<kActSoftmax>(t * C::BS, reinterpret_cast<float (*)[64]>(dst + BC::STAGE), lane);
  };

  // dQ of query tile t from the dS tiles (published by the barrier that ended
  // t's iteration), in two parts: the contraction (LDS reads and MFMAs, done
  // while no tile load is in flight) and the atomic adds (issued after the
  // next tile's loads, so that the wait for those loads can leave them in
  // flight). A wave takes the 32-column blocks wave, wave + 4, ...
  constexpr int MAXIT = (C::ITEMS + 3) / 4;
  struct DqWork {
    f32x16 acc[MAXIT];
    int r0;
  };
  // read offsets of this wave's column blocks (wave, wave + 4, ...; those of
  // the first distribution follow the second's)
  DqOffsets dqo[MAXIT];
#pragma unroll
  for (int m = 0; m < MAXIT; ++m) {
    const int it = wave + 4 * m;
    if (C::WANT_B && it < C::NCB_B) dqo[m] = dq_offsets<C::CB>(lane, it);
    else if constexpr (C::WANT_A) dqo[m] = dq_offsets<C::CA>(lane, it - C::NCB_B);
  }
  auto dq_compute = [&](int t, DqWork& w) {
    w.r0 = t * C::BS;
    const int qlast = min(w.r0 + C::BS, NQ) - 1;
    int kmax = blast;
    if (CAUSAL) kmax = min(kmax, qlast + off);
    const int jend = kmax < kb0 ? 0 : (kmax - kb0) / 16 + 1;   // 16-key groups any row of the tile sees
#pragma unroll
    for (int m = 0; m < MAXIT; ++m) {
      const int it = wave + 4 * m;
      if (it < C::ITEMS) {
        if (C::WANT_B && it < C::NCB_B)
          w.acc[m] = dq_block_mma<C::CB, C::BR / 16>(ds_b, kres_b, dqo[m], jend);
        else if constexpr (C::WANT_A)
          w.acc[m] = dq_block_mma<C::CA, C::BR / 16>(ds_a, kres_a, dqo[m], jend);
      }
    }
  };
  // Returns how many of this wave's last vector memory instructions are
  // atomics that the next wait may leave in flight: kDqAtomicsPerBlock per
  // item of a full tile, 0 when the tile is partial (some adds masked off,
  // count unknown).
  auto dq_add = [&](const DqWork& w) {
    const int qmin_seen = kb0 - off;   // earlier rows see no key of the block
    const bool full = w.r0 + C::BS <= NQ && (!CAUSAL || w.r0 >= qmin_seen);
    int issued = 0;
#pragma unroll
    for (int m = 0; m < MAXIT; ++m) {
      const int it = wave + 4 * m;
      if (it < C::ITEMS) {
        if (C::WANT_B && it < C::NCB_B) {
          if (dQb) {
            if (full)
              dq_block_add<DB, CAUSAL, true>(w.acc[m], it, lane, dQb, (size_t)bh * NQ, w.r0, NQ, qmin_seen, sb);
            else
              dq_block_add<DB, CAUSAL, false>(w.acc[m], it, lane, dQb, (size_t)bh * NQ, w.r0, NQ, qmin_seen, sb);
            issued += kDqAtomicsPerBlock;
          }
        } else if constexpr (C::WANT_A) {
          if (dQa) {
            if (full)
              dq_block_add<DA, CAUSAL, true>(w.acc[m], it - C::NCB_B, lane, dQa, (size_t)bh * NQ, w.r0, NQ,
                                             qmin_seen, sa);
            else
              dq_block_add<DA, CAUSAL, false>(w.acc[m], it - C::NCB_B, lane, dQa, (size_t)bh * NQ, w.r0, NQ,
                                              qmin_seen, sa);
            issued += kDqAtomicsPerBlock;
          }
        }
      }
    }
    return full ? issued : 0;
  };

  // One tile: cur holds query tile t and sstat[buf] its statistics; the next
  // tile (if any) is loaded into nxt meanwhile. prev is the tile whose dS
  // tiles are in LDS (-1 on the first step).
  auto step = [&](const u32x4* cur, u32x4* nxt, int i, int buf, int prev) {
    const int ln = opaque(lane);
    const int t = tile_at(i);
    const bool has_next = i + 1 < nt;
    // the previous tile's dQ: contraction first, atomics after the next
    // tile's loads
    DqWork w;
    if (prev >= 0) dq_compute(prev, w);
    if (has_next) stage_in(tile_at(i + 1), nxt);
    // The end-of-tile wait below leaves the newest kDqAtomicsPerBlock vector
    // memory instructions in flight. That is safe only because every one of
    // them is an atomic issued after the last load of the next tile: vector
    // memory instructions complete in issue order, so all loads are done.
    // Nothing may move between the loads and the atomics.
    __builtin_amdgcn_sched_barrier(0);
    const int n_atomic = prev >= 0 ? dq_add(w) : 0;
    __builtin_amdgcn_sched_barrier(0);

    const int r0 = t * C::BS;
    const int qlast = min(r0 + C::BS, NQ) - 1;
    bool active = kw < NK;
    bool need_mask = r0 + C::BS > NQ || kw + 31 >= NK;
    if (CAUSAL) {
      active = active && (qlast + off >= kw);
      need_mask = need_mask || (wklast > r0 + off);
    }
    const f32x4 (&st)[4][C::BS / 4] = sstat[buf];
    auto stats = [&](int e) {
      const int grp = 2 * (e >> 2) + half;
      return RowStats{st[0][grp][e & 3], st[1][grp][e & 3], st[2][grp][e & 3], st[3][grp][e & 3]};
    };
    auto ok = [&](int e) {
      const int q = r0 + 8 * (e >> 2) + 4 * half + (e & 3);
      return q < NQ && myk < NK && (!CAUSAL || myk <= q + off);
    };
    float dsa[16], dsb[16];
    asm volatile("" : "+v"(kres_row));
    if (active) {
      // the general path also takes the tiles whose g could not be folded
      if (opaque(need_mask || !sfold[buf]))
        bwd_dlogits_tile<DA, DB, MODE, true, false, kActSoftmax>(cur, op_a, op_b, ca, cb, sa, sb, ln, stats, ok, dsa,
                                                                 dsb);
      else
        bwd_dlogits_tile<DA, DB, MODE, false, true, kActSoftmax>(cur, op_a, op_b, ca, cb, sa, sb, ln, stats, ok, dsa,
                                                                 dsb);
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) { dsa[e] = 0.f; dsb[e] = 0.f; }
    }
    // the dS tiles are free once every wave has read them for the previous tile's dQ
    if (prev >= 0) barrier_no_fence();
    if constexpr (C::WANT_A) store_ds(ds_a, kloc, half, dsa);
    if constexpr (C::WANT_B) store_ds(ds_b, kloc, half, dsb);
    if (active) bwd_grad_tile<DA, DB, MODE>(cur, dsa, dsb, dka, dkb, tro);
    if (has_next) {
      // vector memory operations complete in issue order: with the newest
      // kDqAtomicsPerBlock (atomics, see above) allowed in flight, the next
      // tile's loads are done
      if (n_atomic >= kDqAtomicsPerBlock) wait_vmem_le<kDqAtomicsPerBlock>();
      else wait_vmem();
      stage_row_stats<C::BS>(raw_of(nxt), tile_at(i + 1) * C::BS, NQ, rdma.has_g, sstat[buf ^ 1], &sfold[buf ^ 1],
                             tid);
    }
    wait_lds();
    barrier_no_fence();
    return t;
  };

  if (nt > 0) {
    stage_in(tile_at(0), st0);
    wait_vmem();
    stage_row_stats<C::BS>(raw_of(st0), tile_at(0) * C::BS, NQ, rdma.has_g, sstat[0], &sfold[0], tid);
  }
  wait_vmem();   // key block copies
  __syncthreads();
  int prev = -1;
  for (int i = 0; i < nt; i += 2) {
    prev = step(st0, st1, i, 0, prev);
    if (i + 1 < nt) prev = step(st1, st0, i + 1, 1, prev);
  }
  if (prev >= 0) {
    DqWork w;
    dq_compute(prev, w);
    dq_add(w);
  }

  if constexpr (C::WANT_B)
    if (dKb) write_grad<DB>(dKb, dkb, (size_t)bh * NK, kw, NK, sb, lane);
  if constexpr (C::WANT_A)
    if (dKa) write_grad<DA>(dKa, dka, (size_t)bh * NK, kw, NK, sa, lane);
}

}  // namespace streamkl
