// Shared device helpers of the gfx950 attention-KL kernels: vector types,
// the bf16 MFMA, the LDS tile layout and the workgroup -> tile mapping.
//
// Layout facts relied on throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   A operand (32 x 16):  lane l holds A[l % 32][8 * (l / 32) + 0..7]
//   B operand (16 x 32):  lane l holds B[8 * (l / 32) + 0..7][l % 32]
//   C result  (32 x 32):  lane l, register i holds C[8 * (i / 4) + 4 * (l / 32) + i % 4][l % 32]
// ds_read_b64_tr_b16 (gfx950): within each group of 16 lanes, lane i receives
//   element (i % 4) of the 8-byte pieces addressed by lanes 4 * t + i / 4,
//   t = 0..3, so four lanes pointing at four rows of a row-major matrix
//   deliver one column of those rows to each receiving lane.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace streamkl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));   // one 16-byte chunk
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) char lds_char;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kNegInf = -__builtin_inff();
constexpr int kXcds = 8;        // MI355X: 8 accelerator complex dies, 32 CUs each
constexpr int kThreads = 256;   // threads of a 4-wave workgroup

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 2^x on the transcendental unit (v_exp_f32); exp2(-inf) = 0.
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// What the sigmoid-score divergence needs of the two scaled logits za, zb
// (z = S log2(e)) of one (row, key) pair: A = sigmoid(S), 1 - A = sigmoid(-S)
// for both, and lr = log2(A_a / A_b). With e = 2^-|z| in (0, 1] and
// w = 1 + e, A = 1/w or e/w and -log2 A = max(-z, 0) + log2 w, so
//   lr = max(-zb, 0) - max(-za, 0) + log2(w_b / w_a),
//   w_b / w_a = 1 + (e_b - e_a) / w_a:
// one log2, with the reciprocal 1/w_a already formed for A_a, where the two
// logarithms taken separately would cost a second transcendental; written
// as 1 + (e_b - e_a)/w_a the ratio is exactly 1 for equal logits, so equal
// score rows give lr = 0 exactly. Nothing overflows and 1 - A is no
// cancellation. A masked stand-in logit (-1e30) gives A = 0, 1 - A = 1 and a
// finite lr.
// The terms of one logit alone, for gradients that need no logarithm:
// a = sigmoid(S), na = 1 - a.
struct SigmoidTerms {
  float a, na;
};
__device__ __forceinline__ SigmoidTerms sigmoid_terms(float z) {
  const float e = __builtin_amdgcn_exp2f(-fabsf(z));
  const float iw = __builtin_amdgcn_rcpf(1.f + e);
  const float ew = e * iw;
  const bool pos = z >= 0.f;
  return SigmoidTerms{pos ? iw : ew, pos ? ew : iw};
}

struct SigmoidPair {
  float a, na;   // A_a, 1 - A_a
  float b, nb;   // A_b, 1 - A_b
  float lr;      // log2(A_a / A_b)
};
__device__ __forceinline__ SigmoidPair sigmoid_pair(float za, float zb) {
  const float ea = __builtin_amdgcn_exp2f(-fabsf(za)), eb = __builtin_amdgcn_exp2f(-fabsf(zb));
  const float wa = 1.f + ea, wb = 1.f + eb;   // in (1, 2]
  const float iwa = __builtin_amdgcn_rcpf(wa), iwb = __builtin_amdgcn_rcpf(wb);
  const float ewa = ea * iwa, ewb = eb * iwb;
  const bool pa = za >= 0.f, pb = zb >= 0.f;
  const float lr = (fmaxf(-zb, 0.f) - fmaxf(-za, 0.f)) + __builtin_amdgcn_logf(__builtin_fmaf(eb - ea, iwa, 1.f));
  return SigmoidPair{pa ? iwa : ewa, pa ? ewa : iwa, pb ? iwb : ewb, pb ? ewb : iwb, lr};
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// ---------------------------------------------------------------------------
// LDS tiles. A tile of R rows x D bf16 is stored as R * (D / 8) 16-byte
// chunks, row after row, with chunk c of row r placed at slot c ^ swz(r).
// The gfx950 LDS serves a 16-byte-per-lane read 16 lanes at a time from 64
// four-byte banks, i.e. 16 chunk slots; a 16-lane group must touch 16
// distinct slots modulo 16. The two read patterns are
//  - MFMA operand rows: 16 consecutive rows at the same chunk, and
//  - transpose reads: 4 consecutive rows (first one a multiple of 4) at
//    4 consecutive chunks (first one a multiple of 4), two 16-lane groups.
// For rows of 16 or 32 chunks (D = 128, 256) slot mod 16 is the chunk's low
// four bits: XOR them with 4 (r mod 4) + (r / 4 mod 4), a bijection over 16
// rows that moves 4 consecutive rows to 4 disjoint aligned chunk quads. For
// rows of 8 or 24 chunks (D = 64, 192) two rows share the 16 slots: XOR the
// low three bits with 4 (r / 2 mod 2) + (r / 4 mod 4), which separates rows
// of equal parity the same way.
// ---------------------------------------------------------------------------
template <int CPR>
__host__ __device__ constexpr int swz(int r) {
  static_assert(CPR % 8 == 0, "rows must be a multiple of 8 chunks (D a multiple of 64)");
  return (CPR % 16 == 0) ? (4 * (r & 3) + ((r >> 2) & 3)) : (4 * ((r >> 1) & 1) + ((r >> 2) & 3));
}

template <int CPR>
__device__ __forceinline__ int chunk_slot(int r, int c) { return r * CPR + (c ^ swz<CPR>(r)); }

// 8 consecutive bf16 (one chunk) of row r: an MFMA A/B operand.
template <int CPR>
__device__ __forceinline__ bf16x8 lds_row8(const u32x4* tile, int r, int c) {
  return __builtin_bit_cast(bf16x8, tile[chunk_slot<CPR>(r, c)]);
}

// Transpose read at a byte offset of an LDS buffer. In a swizzled tile the
// lane's 4 bf16 at (row r, column e), e a multiple of 4, sit at byte
// chunk_slot(r, e / 8) * 16 + ((e / 4) % 2) * 8; see the layout note at the
// top of this file.
__device__ __forceinline__ bf16x4 lds_tr4_at(const void* buf, int byte) {
  const lds_char* base = (const lds_char*)(buf);
  i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + byte));
  return __builtin_bit_cast(bf16x4, v);
}

__device__ __forceinline__ bf16x8 cat8(const bf16x4& lo, const bf16x4& hi) {
  bf16x8 r;
#pragma unroll
  for (int t = 0; t < 4; ++t) { r[t] = lo[t]; r[t + 4] = hi[t]; }
  return r;
}

// 8 fp32 -> 8 bf16 (round to nearest even), registers first .. first + 7.
__device__ __forceinline__ bf16x8 pack8(const float* v) {
  bf16x8 r;
#pragma unroll
  for (int t = 0; t < 8; ++t) r[t] = (__bf16)v[t];
  return r;
}

// ---------------------------------------------------------------------------
// Tile staging by direct-to-LDS buffer loads (buffer_load_dwordx4 ... lds).
// A buffer resource covers one [N, D] bf16 matrix of one (batch, head); reads
// past its end return zeros, so ragged tails need no clamping (the kernels
// mask those rows). One such load moves 64 x 16 bytes and writes them to LDS
// at M0 + 16 * lane: wave w's i-th load fills chunk slots
// 256 i + 64 w + lane of the stage, and each lane fetches whichever (row,
// chunk) the swizzled layout stores in its slot. No VGPR holds tile data.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // dword 3 = 0x00020000: raw (untyped) 32-bit data format, as used for gfx9 raw buffer access
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// s_waitcnt vmcnt(N) with expcnt and lgkmcnt left unconstrained (gfx9
// encoding: vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void wait_vmem_le() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit counter");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
__device__ __forceinline__ void wait_vmem() { wait_vmem_le<0>(); }

// v, in a register the compiler cannot see through. Tile loops unrolled over
// two stage arrays pass the lane index through this once per tile, so that
// the compiler computes each copy's LDS addresses when it needs them rather
// than all of them up front (holding them in registers); the stage bases
// stay plain array addresses, which the compiler's alias tracking needs.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// fp32 atomic add to global memory, result unused (global_atomic_add_f32).
// The pointer is cast to the global address space: through a generic pointer
// the compiler would have to assume the add may write LDS and would wait for
// it before every later LDS access.
typedef __attribute__((address_space(1))) float global_float;
__device__ __forceinline__ void atomic_add_global(float* p, float v) {
#if defined(__HIP_DEVICE_COMPILE__)
  [[clang::atomic(no_remote_memory, no_fine_grained_memory, ignore_denormal_mode)]] {
    __hip_atomic_fetch_add((global_float*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
#endif
}

// s_waitcnt lgkmcnt(0) alone: this wave's LDS accesses have completed.
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier without a memory fence. __syncthreads() also releases and
// acquires memory, which on gfx950 waits for every outstanding vector memory
// operation of the wave, the tile loads still streaming into LDS included,
// and so would drain the load pipeline at every barrier. The ring protocols
// here do not need that: before a barrier that publishes a stage, the waves
// that loaded it wait for exactly those loads (wait_vmem_le), and every LDS
// read of a stage has returned before the barrier that lets it be refilled
// (its value has been consumed). The signal fences keep the compiler from
// moving memory accesses across the barrier, the scheduling barriers keep it
// from moving any instruction across (phases stay where the code puts them).
__device__ __forceinline__ void barrier_no_fence() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Head dims that are not a multiple of 64 (32, 96, 160, 224) run the kernels
// of the next multiple of 64: in LDS and in registers a row keeps its
// compile-time width, and the chunks past the row's real length are zeros.
// A staging lane whose chunk lies past the real length points its load at
// kOutOfSlab, an offset beyond every slab (a bf16 slab of one head is below
// 2^31 bytes, and tile offsets stay below 2^31 too, so the sum does not
// wrap): the buffer range check turns the load into zeros.
constexpr uint32_t kOutOfSlab = 0x80000000u;

// Byte offset of logical chunk c of tile row r in a global slab whose rows
// hold creal 16-byte chunks, or kOutOfSlab for a padding chunk.
__device__ __forceinline__ uint32_t slab_chunk_offset(int r, int c, int creal) {
  return c < creal ? (uint32_t)(r * creal + c) * 16u : kOutOfSlab;
}

// CB = 0 stages rows of a single matrix. creal_a, creal_b: 16-byte chunks
// per row in global memory (CA, CB unless the head dim is padded).
template <int R, int CA, int CB, int NT = kThreads>
struct TileDma {
  static constexpr int NCH = R * (CA + CB) / NT;
  static constexpr int NCH_A = R * CA / NT;
  static_assert((R * (CA + CB)) % NT == 0 && (R * CA) % NT == 0, "staging split");
  static_assert(CB == 0 || NCH > NCH_A, "second matrix");
  uint32_t voff[NCH];   // byte offset (from the tile's first row) of the chunk this lane fetches

  __device__ __forceinline__ explicit TileDma(int tid, int creal_a = CA, int creal_b = CB) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int p = tid + NT * i;
      if (i < NCH_A) {
        const int r = p / CA, c = (p - r * CA) ^ swz<CA>(r);
        voff[i] = slab_chunk_offset(r, c, creal_a);
      } else if constexpr (CB > 0) {
        const int pp = p - R * CA;
        const int r = pp / CB, c = (pp - r * CB) ^ swz<CB>(r);
        voff[i] = slab_chunk_offset(r, c, creal_b);
      }
    }
  }

  // Rows row0 .. row0 + R - 1 of A and B into `stage` (R * (CA + CB) chunks);
  // dra, drb: the rows' lengths in global memory (elements). The row offset
  // goes into the per-lane offset, which the buffer range check covers (the
  // scalar offset is not range checked).
  __device__ __forceinline__ void issue(rsrc_t ra, rsrc_t rb, int row0, u32x4* stage, int wave, int dra = 8 * CA,
                                        int drb = 8 * CB) const {
#if defined(__HIP_DEVICE_COMPILE__)   // the host pass never runs this; keep its builtins out of it
    const uint32_t base_a = (uint32_t)row0 * (uint32_t)dra * 2u, base_b = (uint32_t)row0 * (uint32_t)drb * 2u;
#pragma unroll
    for (int i = 0; i < NCH_A; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(stage + NT * i + 64 * wave), 16,
                                               voff[i] + base_a, 0, 0, 0);
#pragma unroll
    for (int i = NCH_A; i < NCH; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(stage + NT * i + 64 * wave), 16,
                                               voff[i] + base_b, 0, 0, 0);
#endif
  }
};

// ---------------------------------------------------------------------------
// Row-padded tile layout (forward key tiles). Each row of CPR chunks gets P
// slots; its chunks sit in the order 0, 2, 4, ..., 1, 3, 5, ... from slot
// rot(r) of the row. An MFMA operand lane of row r reads chunks 2 ks + half,
// ks = 0, 1, ...: in this layout they are contiguous from
// base(r, half) = r P + rot(r) + half CPR / 2, so one base register and
// immediate offsets address all of them. P = 8 (mod 16) and rot(r) =
// (r / 2) mod 8 put 16 consecutive rows at one position into 16 distinct
// groups of four banks (the read is conflict-free); the remaining P - CPR
// slots of a row are padding.
// ---------------------------------------------------------------------------
template <int CPR>
struct PadRows {
  static constexpr int P = CPR <= 16 ? 24 : 40;
  static_assert(CPR % 8 == 0 && CPR <= 32, "rows of 8 to 32 chunks");
  __host__ __device__ static constexpr int rot(int r) { return (r >> 1) & 7; }
  __host__ __device__ static constexpr int base(int r, int half) { return r * P + rot(r) + half * (CPR / 2); }
};

// Direct-to-LDS staging of R rows of A (CA chunks) and B (CB chunks) into the
// row-padded layout (R P_A + R P_B slots). Slot s of a tensor holds row
// s / P, position p = s mod P - rot(row); positions outside 0 .. CPR - 1 are
// padding and reload the row's first chunk.
template <int R, int CA, int CB, int NT>
struct PadTileDma {
  static constexpr int PA = PadRows<CA>::P, PB = PadRows<CB>::P;
  static constexpr int NCH_A = R * PA / NT, NCH = NCH_A + R * PB / NT;
  static_assert((R * PA) % NT == 0 && (R * PB) % NT == 0, "staging split");
  uint32_t voff[NCH];

  template <int CPR, int P>
  __device__ __forceinline__ static uint32_t chunk_of(int s, int creal) {
    const int r = s / P, p = s - r * P - PadRows<CPR>::rot(r);
    const int c = (p < 0 || p >= CPR) ? 0 : (p < CPR / 2 ? 2 * p : 2 * (p - CPR / 2) + 1);
    return slab_chunk_offset(r, c, creal);
  }
  __device__ __forceinline__ explicit PadTileDma(int tid, int creal_a = CA, int creal_b = CB) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int p = tid + NT * i;
      voff[i] = i < NCH_A ? chunk_of<CA, PA>(p, creal_a) : chunk_of<CB, PB>(p - R * PA, creal_b);
    }
  }
  __device__ __forceinline__ void issue(rsrc_t ra, rsrc_t rb, int row0, u32x4* stage, int wave, int dra = 8 * CA,
                                        int drb = 8 * CB) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t base_a = (uint32_t)row0 * (uint32_t)dra * 2u, base_b = (uint32_t)row0 * (uint32_t)drb * 2u;
#pragma unroll
    for (int i = 0; i < NCH_A; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(stage + NT * i + 64 * wave), 16,
                                               voff[i] + base_a, 0, 0, 0);
#pragma unroll
    for (int i = NCH_A; i < NCH; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(stage + NT * i + 64 * wave), 16,
                                               voff[i] + base_b, 0, 0, 0);
#endif
  }
};

// ---------------------------------------------------------------------------
// Workgroup -> tile mapping. The dispatcher hands workgroup w to XCD w % 8,
// and each XCD has its own L2. Renumber so that XCD x receives a contiguous
// range of logical tiles: the workgroups resident on one XCD then belong to
// the same (batch, head) and stream the same key tiles through its L2.
// Bijective for any grid size.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int xcd_logical(int bid, int nb) {
  const int q = nb / kXcds, r = nb % kXcds;
  const int x = bid % kXcds, k = bid / kXcds;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + k;
}

// ---------------------------------------------------------------------------
// Causal grids. Under the causal mask the work of a head's blocks falls
// linearly from its longest block to its shortest (query block t of T sees
// about t + 1 key blocks; key block t is seen by about T - t query blocks).
// Handed out head by head, an XCD starts the long and the short blocks of its
// first heads together and the long blocks of its last heads late; a grid of
// a few rounds of workgroups then finishes unevenly. causal_block keeps each
// XCD's contiguous range of heads but hands out that range rank by rank: the
// longest block of each of its heads, then the second longest of each, and
// so on, so that the blocks dispatched into slots freed later are ever
// shorter (longest processing time first). Grids of many rounds balance
// themselves in head order, and there the workgroups resident on an XCD
// stream the same head's tiles through its L2, which the rank order gives
// up: measured, the rank order took 22% off all three kernels of a 32-head
// 4K causal grid (two rounds) and 8% off a 16K forward (four rounds), and
// added 5% to a 64K key-block grid (32 rounds). So it applies up to
// kRankOrderMaxRounds rounds of `slots` resident workgroups.
// Sets the head bh and the rank (0 = longest) of workgroup bid of a grid of
// nb = heads * T; when the heads do not split evenly over the XCDs, or the
// grid is longer, the head-by-head order of xcd_logical. Bijective.
// ---------------------------------------------------------------------------
constexpr int kCus = 256;                 // MI355X compute units
constexpr int kRankOrderMaxRounds = 4;

__device__ __forceinline__ void causal_block(int bid, int nb, int T, int slots, int& bh, int& rank) {
  const int heads = nb / T;
  if (heads % kXcds == 0 && nb <= kRankOrderMaxRounds * slots) {
    const int hx = heads / kXcds;   // heads per XCD
    const int x = bid % kXcds, k = bid / kXcds;
    bh = x * hx + k % hx;
    rank = k / hx;
  } else {
    const int l = xcd_logical(bid, nb);
    bh = l / T;
    rank = l - bh * T;
  }
}

// Head and block of this workgroup in a grid of heads * T blocks of a
// kernel that keeps WG_PER_CU workgroups resident per CU: causal grids by
// causal_block (rank 0 = the longest block), others in xcd_logical order.
template <bool CAUSAL, int WG_PER_CU>
__device__ __forceinline__ void head_block(int T, int& bh, int& rank) {
  if (CAUSAL) {
    causal_block(blockIdx.x, gridDim.x, T, kCus * WG_PER_CU, bh, rank);
  } else {
    const int l = xcd_logical(blockIdx.x, gridDim.x);
    bh = l / T;
    rank = l - bh * T;
  }
}

}  // namespace streamkl
