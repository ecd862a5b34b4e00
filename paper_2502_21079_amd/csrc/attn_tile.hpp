// Tile-level building blocks shared by the attention and block-mass kernels
// (gfx950): bounds-checked global->LDS tile loads, the transposed-score MFMA
// tile, online-softmax pieces and the P V update.
//
// Orientation.  Scores are formed transposed, S^T[key][query] = K Q^T, with K
// as the MFMA A operand (read from LDS) and a 32-query Q fragment as the B
// operand (kept in registers).  In the 32x32 accumulator each lane then holds
// 16 keys of ONE query, so the softmax row statistics are lane-local plus one
// exchange between the two half-waves.  The probabilities P^T are already laid
// out as the B operand of the second product O^T[d][query] += V^T P^T, once
// the 16 keys of each MFMA step are ordered to match the accumulator rows; the
// V^T operand is read from a row-major V tile with the LDS transpose read.
//
// Online softmax.  Probabilities are taken against a per-row reference that
// moves only when a row's running sum grows too large, so neither a per-tile
// maximum nor a rescale of the output accumulator is needed for almost every
// tile; the final normalisation uses the same reference, so the result is
// unchanged.  The running sums are formed on the matrix pipe (RowSums).
#pragma once

#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace adaspa {

constexpr int KT = 64;          // keys per tile

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

// Buffer resource words (base, stride 0, size in bytes, the format word of
// make_rsrc) in scalar registers, for the loads issued by dma16.
__device__ __forceinline__ u32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t b = (uint64_t)base;
  u32x4 r;
  r.x = __builtin_amdgcn_readfirstlane((uint32_t)b);
  r.y = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  r.z = __builtin_amdgcn_readfirstlane(bytes);
  r.w = 0x00020000u;
  return r;
}

// One 16-byte-per-lane direct load into LDS: lane l's 16 bytes at voff +
// soff of the buffer go to LDS byte lds + OFS + 16 l.  It is issued as inline
// asm so that the compiler does not track it: otherwise it makes every later
// LDS read wait for the load (vmcnt) unless it can prove the two touch
// different addresses, which it cannot for the ring slots.  The ordering is
// explicit instead: a loaded tile is read only after a vmcnt(0) wait and a
// barrier, and a slot is refilled only after the barrier that follows its
// last read.  M0 carries the LDS address; the compiler sets M0 itself before
// each of its own uses, so clobbering it here is harmless.  The add that
// forms M0 also sets SCC, which is declared clobbered too (a compare whose
// result the compiler kept in SCC across the load would otherwise be lost).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
template <int OFS>
__device__ __forceinline__ void dma16(u32x4 rsrc, uint32_t lds, uint32_t voff, uint32_t soff) {
  asm volatile("s_add_u32 m0, %0, %4\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds), "v"(voff), "s"(rsrc), "s"(soff), "n"(OFS) : "m0", "scc");
}
#pragma clang diagnostic pop

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}

// One [KT, D] bf16 tile in LDS with padded rows: row r starts at chunk
// r * S (16-byte chunks, S = D/8 + PADC).  The K tile has one pad chunk per
// row, so 8 (or 16) consecutive rows read at the same column fall in distinct
// banks; the V tile has two, so each group of 4 rows x 32 bytes read by a
// transposed load covers distinct banks.  With constant strides every operand
// address is one lane base plus a compile-time offset.
template <int D, int NW, int PADC>
struct TileDMA {
  static constexpr int CPR = D / 8;                 // data chunks per row
  static constexpr int S = CPR + PADC;              // chunks per LDS row
  static constexpr int SLOTS = KT * S;              // chunk slots per tile
  static constexpr int NINST = SLOTS / 64;          // 64-slot DMA instructions
  static_assert(SLOTS % 64 == 0, "tile slots must fill whole instructions");
  static constexpr int ELEMS = SLOTS * 8;           // bf16 elements per tile

  // Issue the loads of rows [kbase, kbase + KT).  Rows past the buffer's end
  // and pad slots use an out-of-range offset: the load is skipped and the slot
  // reads zero.
  __device__ __forceinline__ static void issue(__amdgpu_buffer_rsrc_t r, u16* dst, int kbase,
                                               int wave, int lane) {
#pragma unroll
    for (int i0 = 0; i0 < NINST; i0 += NW) {
      const int i = i0 + wave;
      if (i < NINST) {
        const int p = i * 64 + lane;
        const int row = p / S, ch = p % S;
        const uint32_t off = ch < CPR ? (uint32_t)((kbase + row) * D + ch * 8) * 2u : 0xFFFFFFF0u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + i * 64 * 8), 16, off, 0, 0, 0);
      }
    }
  }

  // Issue the loads of a dual tile: rows [0, 32) from keys [ka, ka + 32),
  // rows [32, 64) from keys [kb, kb + 32) (both inside the sequence).  Pad
  // slots use an out-of-range offset: the load is skipped.
  __device__ __forceinline__ static void issue_dual(__amdgpu_buffer_rsrc_t r, u16* dst, int ka, int kb,
                                                    int wave, int lane) {
#pragma unroll
    for (int i0 = 0; i0 < NINST; i0 += NW) {
      const int i = i0 + wave;
      if (i < NINST) {
        const int p = i * 64 + lane;
        const int row = p / S, ch = p % S;
        const int key = row < 32 ? ka + row : kb + (row - 32);
        const uint32_t off = ch < CPR ? (uint32_t)(key * D + ch * 8) * 2u : 0xFFFFFFF0u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + i * 64 * 8), 16, off, 0, 0, 0);
      }
    }
  }

  // Byte offset, inside the tile, of the chunk that slot i * 64 + lane loads
  // when every row of the tile lies inside the sequence.  A pad slot loads a
  // copy of its row's last data chunk (it is never read, and an in-range
  // duplicate keeps every offset below 2^16).
  __device__ __forceinline__ static uint32_t rel_offset(int i, int lane) {
    const int p = i * 64 + lane;
    const int row = p / S, ch = p % S;
    return (uint32_t)(row * D + (ch < CPR ? ch : CPR - 1) * 8) * 2u;
  }
  // Instruction i of a full tile whose first byte is tile_byte: the offset
  // inside the tile comes from rel_offset, the tile start is the scalar
  // offset, so an issue costs no address arithmetic.
  __device__ __forceinline__ static void issue_full(__amdgpu_buffer_rsrc_t r, u16* dst,
                                                    uint32_t tile_byte, int i, uint32_t rel) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + i * 64 * 8), 16, rel,
                                             (int)tile_byte, 0, 0);
  }
};
using std::integral_constant;

// Loads of one full K tile per step (the block-mass pass), uniform over the
// waves as in KVLoader below: wave w issues the tile's DMA instructions
// j * NW + w, j = 0 .. PW-1, and repeats its entry of j - 1 where the list
// runs out, so no load sits behind a branch.
template <int D, int NW>
struct KLoader {
  using K = TileDMA<D, NW, 1>;
  static constexpr int PW = (K::NINST + NW - 1) / NW;
  static_assert(K::NINST >= NW, "a repeated entry must be a load of the same wave");
  uint32_t rel[PW];          // per lane: in-tile source offset of load j
  uint32_t wbase, wlast;     // LDS byte offsets of this wave's pieces of entries 0 and PW-1

  __device__ __forceinline__ void init(int wave, int lane) {
    wbase = (uint32_t)wave * 1024u;
    wlast = wbase - (((PW - 1) * NW + wave >= K::NINST) ? (uint32_t)NW * 1024u : 0u);
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      int f = j * NW + wave;
      if (f >= K::NINST) f -= NW;
      rel[j] = K::rel_offset(f, lane);
    }
  }
  // Load n (a constant once the caller's loop is unrolled) of the tile whose
  // first byte is kbyte into the tile at LDS byte address tile.
  template <int J = 0>
  __device__ __forceinline__ void issue_n(int n, uint32_t tile, u32x4 rK, uint32_t kbyte) const {
    if constexpr (J < PW) {
      if (n == J) dma16<J * NW * 1024>(rK, tile + (J == PW - 1 ? wlast : wbase), rel[J], kbyte);
      else issue_n<J + 1>(n, tile, rK, kbyte);
    }
  }
};


// Loads of one full K tile and one full V tile per step into one ring slot
// laid out [K tile | V tile].  The 64-slot DMA instructions of the two tiles
// form one list of NTOT = K::NINST + V::NINST entries, entry f writing the
// f-th 1 KB piece of the slot, and wave w issues entry j * NW + w for j = 0
// .. PW-1.  Every wave issues the same number of loads and none sits behind
// a branch: where the list runs out (the last j of some waves) a wave repeats
// its entry of j - 1 (the same data to the same place).  The source of a load
// is the tile's first byte (scalar offset) plus a per-lane in-tile offset kept
// in a register, and its destination the slot plus a per-wave constant.
// Entries j with (j+1)*NW <= K::NINST are K loads for every wave, entries
// with j*NW >= K::NINST are V loads for every wave, and the one j in between
// (if any) is K for some waves and V for the others ("mixed").
template <int D, int NW>
struct KVLoader {
  using K = TileDMA<D, NW, 1>;
  using V = TileDMA<D, NW, 2>;
  static constexpr int NK = K::NINST;
  static constexpr int NTOT = K::NINST + V::NINST;
  static constexpr int PW = (NTOT + NW - 1) / NW;           // loads per wave and step
  static constexpr int ELEMS = K::ELEMS + V::ELEMS;         // bf16 elements per ring slot
  static constexpr int VOFF = K::ELEMS;                     // V tile within the slot
  static_assert(K::ELEMS == NK * 512, "the V tile starts right after the K tile's pieces");
  static_assert(V::NINST >= NW, "a repeated entry must be a V load of the same wave");
  static_assert(NK % NW == 0 || NK / NW != PW - 1, "the mixed entry is not the last one");
  static_assert(KT * D * 2 <= 65536, "in-tile offsets must fit in 16 bits");
  static constexpr bool all_k(int j) { return (j + 1) * NW <= NK; }
  static constexpr bool all_v(int j) { return j * NW >= NK; }

  uint32_t rel[PW];          // per lane: in-tile source offset of load j
  uint32_t wbase;            // LDS byte offset of this wave's piece of entry j = 0
  uint32_t wlast;            // the same for the last entry (one row of pieces lower if it repeats)
  bool mixed_v;              // the mixed entry is a V load for this wave

  __device__ __forceinline__ void init(int wave, int lane) {
    wbase = (uint32_t)wave * 1024u;
    wlast = wbase - (((PW - 1) * NW + wave >= NTOT) ? (uint32_t)NW * 1024u : 0u);
    mixed_v = (NK / NW) * NW + wave >= NK;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      int f = j * NW + wave;
      if (f >= NTOT) f -= NW;
      rel[j] = f < NK ? K::rel_offset(f, lane) : V::rel_offset(f - NK, lane);
    }
  }
  // Load J of this wave into the slot at LDS byte address slot; rK / rV are
  // the K and V resources and rM the one of this wave's mixed entry, kbyte /
  // vbyte / mbyte the first bytes of the K tile, the V tile and the mixed
  // entry's tile.
  template <int J>
  __device__ __forceinline__ void issue(uint32_t slot, u32x4 rK, u32x4 rV, u32x4 rM, uint32_t kbyte,
                                        uint32_t vbyte, uint32_t mbyte) const {
    constexpr int F = J * NW * 1024;
    if constexpr (J == PW - 1) dma16<F>(rV, slot + wlast, rel[J], vbyte);
    else if constexpr (all_k(J)) dma16<F>(rK, slot + wbase, rel[J], kbyte);
    else if constexpr (all_v(J)) dma16<F>(rV, slot + wbase, rel[J], vbyte);
    else dma16<F>(rM, slot + wbase, rel[J], mbyte);
  }
  // Load n (a constant once the caller's loop is unrolled).
  template <int J = 0>
  __device__ __forceinline__ void issue_n(int n, uint32_t slot, u32x4 rK, u32x4 rV, u32x4 rM, uint32_t kbyte,
                                          uint32_t vbyte, uint32_t mbyte) const {
    if constexpr (J < PW) {
      if (n == J) issue<J>(slot, rK, rV, rM, kbyte, vbyte, mbyte);
      else issue_n<J + 1>(n, slot, rK, rV, rM, kbyte, vbyte, mbyte);
    }
  }

  // Dual slots: rows [0, 32) of the K and V tiles come from one 32-key half
  // tile, rows [32, 64) from another.  Bit j of the returned mask is set when
  // this lane's load j fills a row of the second half (the pieces and their
  // assignment to the waves are those above).
  __device__ __forceinline__ static uint32_t half_mask(int wave, int lane) {
    uint32_t m = 0;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      int f = j * NW + wave;
      if (f >= NTOT) f -= NW;
      const int row = f < NK ? (f * 64 + lane) / K::S : ((f - NK) * 64 + lane) / V::S;
      if (row >= 32) m |= 1u << j;
    }
    return m;
  }
  // Load J of a dual slot: ka / va are the first bytes of the first half's
  // K / V keys, kb / vb those of the second half's minus 32 rows (the in-tile
  // offsets of its rows start at row 32), and the lane adds the one of the
  // half its row belongs to; the scalar offset is zero.
  template <int J>
  __device__ __forceinline__ void issue_dual(uint32_t slot, u32x4 rK, u32x4 rV, u32x4 rM, uint32_t ka,
                                             uint32_t kb, uint32_t va, uint32_t vb, uint32_t hmask) const {
    constexpr int F = J * NW * 1024;
    const bool second = (hmask >> J) & 1u;
    const uint32_t kk = second ? kb : ka, vv = second ? vb : va;
    if constexpr (J == PW - 1) dma16<F>(rV, slot + wlast, rel[J] + vv, 0u);
    else if constexpr (all_k(J)) dma16<F>(rK, slot + wbase, rel[J] + kk, 0u);
    else if constexpr (all_v(J)) dma16<F>(rV, slot + wbase, rel[J] + vv, 0u);
    else dma16<F>(rM, slot + wbase, rel[J] + (mixed_v ? vv : kk), 0u);
  }
  template <int J = 0>
  __device__ __forceinline__ void issue_dual_n(int n, uint32_t slot, u32x4 rK, u32x4 rV, u32x4 rM, uint32_t ka,
                                               uint32_t kb, uint32_t va, uint32_t vb, uint32_t hmask) const {
    if constexpr (J < PW) {
      if (n == J) issue_dual<J>(slot, rK, rV, rM, ka, kb, va, vb, hmask);
      else issue_dual_n<J + 1>(n, slot, rK, rV, rM, ka, kb, va, vb, hmask);
    }
  }
};

// The K or V part of the ring slots: part[b] is the tile in slot b.
template <int ELEMS, int OFF>
struct SlotPart {
  u16 (*slots)[ELEMS];
  __device__ __forceinline__ u16* operator[](int b) const { return slots[b] + OFF; }
};

// Maximum without the sNaN canonicalisation that fmaxf needs in IEEE mode
// (a NaN score propagates, which is fine: the row is then NaN either way).
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Keeps the computation of v at this point of the instruction stream: the
// empty volatile asm is ordered with the scheduling fences around it, so the
// compiler can neither sink the work that produces v past them (out of the
// MFMA slot it was placed in) nor hoist it.
__device__ __forceinline__ void pin(float& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void pin(bf16x2& v) { asm volatile("" : "+v"(v)); }

__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)

template <int D>
__device__ __forceinline__ void load_q(const u16* qh, int qrow, int L, int hw, bf16x8 (&qf)[D / 16]) {
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    if (qrow < L)
      qf[ks] = *reinterpret_cast<const bf16x8*>(qh + (size_t)qrow * D + ks * 16 + hw * 8);
    else
      qf[ks] = bf16x8{};
  }
}

// S^T tile for G groups of 32 keys (G = 2: a 64-key tile; G = 1: its first
// 32 keys): lane (hw, c32) gets keys 32g + 8(e/4) + 4hw + e%4 of query c32 in
// s[g][e].
template <int D, int S, int G = 2>
__device__ __forceinline__ void qk_tile(const u16* sK, const bf16x8 (&qf)[D / 16], int c32, int hw,
                                        f32x16 (&s)[2]) {
  const u16* base = sK + (c32 * S + hw) * 8;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    s[g] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      bf16x8 kf = *reinterpret_cast<const bf16x8*>(base + (32 * g * S + 2 * ks) * 8);
      s[g] = mfma32(kf, qf[ks], s[g]);
    }
  }
}

__device__ __forceinline__ void mask_tile(f32x16 (&s)[2], int kvalid, int hw) {
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = 32 * g + 8 * (e >> 2) + 4 * hw + (e & 3);
      if (key >= kvalid) s[g][e] = -INFINITY;
    }
}

template <int NCH>
__device__ __forceinline__ void zero_lds(u16* p, int tid, int nt) {
  for (int i = tid; i < NCH; i += nt) *reinterpret_cast<u32x4*>(p + i * 8) = u32x4{0, 0, 0, 0};
}

// Online softmax against a lazy reference.  Probabilities of a row are taken
// as exp2(s * sl2 - mc) with mc = m * sl2 for a reference m (raw score units)
// that is NOT the running maximum, so no per-tile maximum is computed on the
// common path; the final normalisation uses the same reference, so the
// result is the softmax whatever the reference.  The first tile with a finite
// score sets it to that tile's maximum, however negative (against mc = 0 a
// row whose scaled scores all lie below the fp32 exponent range would sum to
// zero).  In the pipeline it then moves only when the row's running sum
// passes kRowSumLimit (move_reference below); on the masked, exact path it
// moves when the tile's probabilities, summed over one lane's keys, exceed
// kTileSumLimit (RowRef::lim, checked before the tile enters P V), so there no
// probability exceeds 2^16 whatever the scores.  When the reference moves,
// sums taken against the old one are rescaled.
constexpr float kTileSumLimit = 65536.f;

struct RowRef {
  float m = -INFINITY;   // reference, raw score units; -inf until a finite score is seen
  float mc = 0.f;        // m * sl2 (0 while m is -inf)
  float lim = -1.f;      // tile sum above which the reference must move (below any sum while m is -inf)

  // m <- max(m, row maximum of s) for the rows of this wave (the two
  // half-waves holding a row agree); returns the rescale factor of sums
  // taken against the old reference.
  template <int G = 2>
  __device__ __forceinline__ float raise(const f32x16 (&s)[2], float sl2) {
    float mt = -INFINITY;
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 16; e += 2) mt = vmax(mt, vmax(s[g][e], s[g][e + 1]));
    float lo, hi;
    half_pair(mt, lo, hi);
    mt = vmax(lo, hi);
    const float mnew = fmaxf(m, mt);
    const float a = (mnew == -INFINITY) ? 1.f : fast_exp2((m - mnew) * sl2);
    m = mnew;
    mc = (m == -INFINITY) ? 0.f : m * sl2;
    lim = (m == -INFINITY) ? -1.f : kTileSumLimit;
    return a;
  }
  // Moves a set reference up by d (log2 units): sums taken against the old
  // one scale by 2^-d.
  __device__ __forceinline__ void shift(float d, float sl2) {
    mc += d;
    m = mc / sl2;
  }
};

// Running row sums of the rounded probabilities, formed on the matrix pipe.
// The 16x16x32 bf16 MFMA takes a P^T operand of the P V product as its B
// operand (lane l holds 8 keys of query row l % 32, so output column n
// gathers lanes n, n+16, n+32 and n+48, i.e. rows n and n+16) and a 0/1
// selector as A: output rows 0-7 keep k-groups 0 and 2 (lanes n, n+32:
// row n), output rows 8-15 keep k-groups 1 and 3 (row n+16).  Lane l then
// holds the sum of query row (l % 16) + 16 (l / 32), the same in all four
// accumulator entries.  (A v_dot2c per pair on the VALU holds the matrix
// pipe ~20 cycles each; four of these MFMAs take 64 cycles per step.)
// Sums above kRowSumLimit move the reference by log2 of the sum; a sum above
// kRowSumBad (or not finite) means a single tile jumped so far above the
// reference that a product may have overflowed, and the caller redoes the
// row on the exact path.
constexpr float kRowSumLimit = 1099511627776.f;                   // 2^40
constexpr float kRowSumBad = 1267650600228229401496703205376.f;   // 2^100

struct RowSums {
  f32x4 acc;
  bf16x8 sel;
  __device__ __forceinline__ void init(int lane) {
    acc = f32x4{0.f, 0.f, 0.f, 0.f};
    const __bf16 v = (((lane & 15) < 8) == (((lane >> 4) & 1) == 0)) ? (__bf16)1.0f : (__bf16)0.0f;
    sel = bf16x8{v, v, v, v, v, v, v, v};
  }
  __device__ __forceinline__ void add(const bf16x8& p) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, p, acc, 0, 0, 0);
  }
  // The sum of query row c32 (the row of the P V layout), from its lane.
  __device__ __forceinline__ static float for_row(float v, int c32) {
    return __shfl(v, c32 < 16 ? c32 : c32 + 16, 64);
  }
};

// P = bf16(exp2(s * sl2 - mc)) for one S^T tile; returns this lane's sum of
// exactly the rounded values that enter P V, so numerator and denominator
// use the same weights.
template <int G = 2>
__device__ __forceinline__ float exp_tile(const f32x16 (&s)[2], float sl2, float mc, bf16x8 (&pb)[2][2]) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float ts = 0.f;
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      const bf16x2 pr = {(__bf16)fast_exp2(fmaf(s[g][e], sl2, -mc)),
                         (__bf16)fast_exp2(fmaf(s[g][e + 1], sl2, -mc))};
      pb[g][e >> 3][e & 7] = pr[0];
      pb[g][e >> 3][(e & 7) + 1] = pr[1];
      ts = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, ts, false);
    }
  return ts;
}

// As exp_tile, and fsum also receives this lane's sum of the unrounded fp32
// exponentials (for block masses, which must not carry the rounding of P).
template <int G = 2>
__device__ __forceinline__ float exp_tile_fsum(const f32x16 (&s)[2], float sl2, float mc, bf16x8 (&pb)[2][2],
                                               float& fsum) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float ts = 0.f, fs = 0.f;
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      const float x0 = fast_exp2(fmaf(s[g][e], sl2, -mc)), x1 = fast_exp2(fmaf(s[g][e + 1], sl2, -mc));
      const bf16x2 pr = {(__bf16)x0, (__bf16)x1};
      pb[g][e >> 3][e & 7] = pr[0];
      pb[g][e >> 3][(e & 7) + 1] = pr[1];
      ts = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, ts, false);
      fs += x0 + x1;
    }
  fsum = fs;
  return ts;
}

// End of a pipelined step (rare branch, taken by the whole wave): rows whose
// running sum (tiles up to the previous one) passed kRowSumLimit move their
// reference up by log2 of the sum, so the sum becomes about 1; rows without a
// reference yet take this tile's maximum (their sums so far are 0).  The sums
// are rescaled here, the output accumulator at the start of the next step
// (pend), and the current tile's probabilities are taken again against the
// new reference.  bad is set when a sum has left the safe range.  A hidden
// tile (block-64 pairs: one the other query block keeps) never sets the
// reference and its probabilities stay exact zeros.
// With BS, *tsum receives the fp32 sum of the retaken probabilities.
template <int G = 2, bool BS = false>
__device__ __forceinline__ void move_reference(RowRef& ref, RowSums& rsum, bool& bad,
                                               const f32x16 (&s_cur)[2], bf16x8 (&p_cur)[2][2],
                                               bool& pend, float& pend_alpha, float sl2, int c32,
                                               bool hidden = false, float* tsum = nullptr) {
  const float sr = rsum.acc[0];
  if (!__any(ref.m == -INFINITY || sr > kRowSumLimit)) return;
  bad = bad || !(sr <= kRowSumBad);
  const float dr = sr > kRowSumLimit ? __builtin_amdgcn_logf(sr) : 0.f;   // log2 of the sum
  const float ar = fast_exp2(-dr);
#pragma unroll
  for (int j = 0; j < 4; ++j) rsum.acc[j] *= ar;
  const float d = RowSums::for_row(dr, c32);        // the same value for this lane's row
  float al;
  if (ref.m == -INFINITY) {
    al = hidden ? 1.f : ref.template raise<G>(s_cur, sl2);
  } else {
    if (d > 0.f) ref.shift(d, sl2);
    al = fast_exp2(-d);
  }
  pend_alpha = al;
  pend = true;
  if constexpr (BS) exp_tile_fsum<G>(s_cur, sl2, hidden ? INFINITY : ref.mc, p_cur, *tsum);
  else exp_tile<G>(s_cur, sl2, hidden ? INFINITY : ref.mc, p_cur);
}

// After the last pipelined tile: its probabilities join the sums, a sum out
// of the safe range sets bad, and the row's sum is returned in the form the
// masked path continues from (the whole sum on the hw = 0 lane of the row, 0
// on the other).
template <int G = 2>
__device__ __forceinline__ float finish_sums(RowSums& rsum, bool& bad, const bf16x8 (&p_last)[2][2],
                                             int hw, int c32) {
#pragma unroll
  for (int j = 0; j < 2 * G; ++j) rsum.add(p_last[j >> 1][j & 1]);
  const float sr = rsum.acc[0];
  bad = bad || !(sr <= kRowSumBad);
  const float v = RowSums::for_row(sr, c32);
  return hw == 0 ? v : 0.f;
}

// Whether every entry of the output accumulator is finite.  The row-sum test
// bounds the probabilities, not their products with V: with large |V| a
// product can overflow fp32 while the sums stay in range, so a non-finite
// accumulator after the pipeline also sends the wave to the exact path (whose
// tile-sum test keeps every probability below 2^16).  The maximum propagates
// NaN, and the comparison fails for NaN and infinity.
template <int ND>
__device__ __forceinline__ bool acc_finite(const f32x16 (&o)[ND]) {
  float m = 0.f;
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int e = 0; e < 16; ++e) m = vmax(m, __builtin_fabsf(o[d][e]));
  return m <= 3.4028234663852886e38f;
}

// Softmax of one tile outside the pipeline (masked tiles): P against the
// current reference, moved first if this tile needs it.  Returns the factor
// by which the output accumulator must be rescaled before this tile's P V
// (1 when the reference did not move); lsum includes the tile afterwards.
__device__ __forceinline__ float softmax_tile(const f32x16 (&s)[2], RowRef& ref, float& lsum, float sl2,
                                              bf16x8 (&pb)[2][2]) {
  float ts = exp_tile(s, sl2, ref.mc, pb);
  float a = 1.f;
  if (__any(ts > ref.lim)) {
    a = ref.raise(s, sl2);
    lsum *= a;
    ts = exp_tile(s, sl2, ref.mc, pb);
  }
  lsum += ts;
  return a;
}

// As softmax_tile; fsum receives this lane's fp32 sum of the tile's
// exponentials against the reference they were finally taken against.
__device__ __forceinline__ float softmax_tile_fsum(const f32x16 (&s)[2], RowRef& ref, float& lsum, float sl2,
                                                   bf16x8 (&pb)[2][2], float& fsum) {
  float ts = exp_tile_fsum(s, sl2, ref.mc, pb, fsum);
  float a = 1.f;
  if (__any(ts > ref.lim)) {
    a = ref.raise(s, sl2);
    lsum *= a;
    ts = exp_tile_fsum(s, sl2, ref.mc, pb, fsum);
  }
  lsum += ts;
  return a;
}

// O^T += V^T P^T for one tile.  MFMA step (g, s2) covers keys
// 32g + 16s2 + 8u + 4hw + j; lane (hw, e) supplies key index 8*(e/4) + 4*hw +
// e%4 of the step.  In each 16-lane group, lane j names row r0 + j/4 and 4
// elements at column d*32 + 16*(grp&1) + 4*(j%4); vlane is that lane's base.
template <int ND, int VS, int G = 2>
__device__ __forceinline__ void pv_tile(const u16* vlane, const bf16x8 (&pb)[2][2], f32x16 (&o)[ND]) {
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const u16* p0 = vlane + (32 * g + 16 * s2) * VS * 8 + d * 32;
        const s16x4 lo = lds_read_tr16(p0);
        const s16x4 hi = lds_read_tr16(p0 + 8 * VS * 8);
        bf16x8 vf;
        __builtin_memcpy(&vf, &lo, 8);
        __builtin_memcpy(reinterpret_cast<char*>(&vf) + 8, &hi, 8);
        o[d] = mfma32(vf, pb[g][s2], o[d]);
      }
}

// Writes one wave's 32 x D output tile (o scaled by inv, rounded to bf16) as
// whole rows: the tile goes through stage, this wave's region of the K/V ring
// (32 rows of D + 8 elements, free once every wave has passed a barrier
// after its last use of the ring), and each store instruction then writes
// 64 / (D / 8) complete rows of 2 D bytes instead of 8-byte pieces of 32
// rows.  Row row0 + r of out gets tile row r; rows at or past L are skipped.
template <int D>
__device__ __forceinline__ void store_rows(const f32x16 (&o)[D / 32], float inv, u16* stage, u16* out,
                                           int row0, int L, int lane) {
  constexpr int ND = D / 32, RS = D + 8, CPR = D / 8, RPI = 64 / CPR;
  const int hw = lane >> 5, c32 = lane & 31;
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bf16x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = (__bf16)(o[d][4 * i + j] * inv);
      *reinterpret_cast<bf16x4*>(stage + c32 * RS + d * 32 + 8 * i + 4 * hw) = w;
    }
#pragma unroll 4
  for (int j = 0; j < 32 / RPI; ++j) {
    const int r = lane / CPR + RPI * j;
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(stage + r * RS + (lane % CPR) * 8);
    if (row0 + r < L) *reinterpret_cast<bf16x8*>(out + (size_t)(row0 + r) * D + (lane % CPR) * 8) = v;
  }
}
template <int D, int NW>
constexpr int kStageElems = NW * 32 * (D + 8);    // ring elements store_rows uses

// One pipelined step, scheduled by hand: NM = 2*NK + 4*ND MFMA slots that
// alternate a QK MFMA (scores of the next tile) and a PV MFMA (output update
// of the previous tile).  The QK MFMAs alternate between the two 32-key score
// groups and the PV MFMAs rotate over the ND output blocks, so two MFMAs into
// the same accumulator are 4 (QK) or 2*ND (PV) slots apart and one wave alone
// keeps the matrix pipe busy; each accumulator still sums in the same order.
// Each slot first issues the LDS operand reads of the slot LA places ahead,
// then its MFMA, then hook(slot) (the caller's tile loads, at most one per
// slot), then its share of the softmax of the current tile against the
// reference mc (below); a scheduling fence closes the slot, so the matrix
// pipe and the VALU work side by side within the wave.  Four slots also add
// the previous tile's rounded probabilities (the operands of its P V) to the
// running row sums: the middle slot of each quarter of the step, or with
// RS_FIRST its first slot, so the last of them is done well before the sum
// test at the end of the step (dense attention: -1%; block-sparse
// attention, whose loads and index picks crowd the first slots, keeps the
// middle).  The sums are the same either way.
// With BS, *tsum receives this lane's sum of the current tile's unrounded
// exponentials, added pair by pair as the pairs are rounded.
template <int D, int KS, int VS, int G = 2, bool BS = false, bool RS_FIRST = false, typename Hook>
__device__ __forceinline__ void pipelined_step(Hook&& hook, const u16* klane, const u16* vlane,
                                               const bf16x8 (&qf)[D / 16], const f32x16 (&s_cur)[2],
                                               const bf16x8 (&p_prev)[2][2], f32x16 (&s_next)[2],
                                               bf16x8 (&p_cur)[2][2], f32x16 (&o)[D / 32], float sl2,
                                               float mc, RowSums& rsum, float* tsum = nullptr) {
  constexpr int NK = D / 16, ND = D / 32;
  constexpr int NQK = G * NK, NPV = 2 * G * ND;      // G score groups of 32 keys
  static_assert(NQK == NPV, "QK and PV slots alternate");
  constexpr int NM = NQK + NPV;
  constexpr int NS = 16 * G;                           // scores per lane
  static_assert(NS % NM == 0 && NM % 2 == 0, "whole exponential pairs per slot pair");
  constexpr int LA = 2;                       // operand lookahead, in slots

  bf16x8 op[NM];
  auto fetch = [&](int i) {
    const int j = i >> 1;
    if ((i & 1) == 0) {       // QK j: g = j % G, ks = j / G
      const int g = j % G, ks = j / G;
      op[i] = *reinterpret_cast<const bf16x8*>(klane + (32 * g * KS + 2 * ks) * 8);
    } else {                  // PV j: d = j % ND, (g, s2) = j / ND
      const int d = j % ND, g = (j / ND) >> 1, s2 = (j / ND) & 1;
      const u16* p0 = vlane + (32 * g + 16 * s2) * VS * 8 + d * 32;
      const s16x4 lo = lds_read_tr16(p0);
      const s16x4 hi = lds_read_tr16(p0 + 8 * VS * 8);
      __builtin_memcpy(&op[i], &lo, 8);
      __builtin_memcpy(reinterpret_cast<char*>(&op[i]) + 8, &hi, 8);
    }
  };
  auto mfma = [&](int i) {
    const int j = i >> 1;
    if ((i & 1) == 0) {
      const int g = j % G, ks = j / G;
      if (ks == 0) s_next[g] = mfma32(op[i], qf[ks], f32x16{});
      else s_next[g] = mfma32(op[i], qf[ks], s_next[g]);
    } else {
      const int d = j % ND, g = (j / ND) >> 1, s2 = (j / ND) & 1;
      o[d] = mfma32(op[i], p_prev[g][s2], o[d]);
    }
  };

  // Slot i owns scores e in [i*PER, (i+1)*PER) of the tile's 32, in (group,
  // element) order.  Their softmax is pipelined over three slots: slot i
  // forms the exponent arguments, slot i+1 takes the exponentials, slot i+2
  // rounds each completed pair to bf16, so no instruction waits on the result
  // of the one just before it.  The last two slots' shares are finished after
  // the MFMAs.
  constexpr int PER = NS / NM;
  constexpr int RSP = NM / (2 * G);           // row-sum MFMAs in slots RS0 + j*RSP
  constexpr int RS0 = RS_FIRST ? 0 : RSP / 2;
  float arg[NS], ex[NS];
  float fs = 0.f;
  auto stage_arg = [&](int i) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = i * PER + u;
      arg[e] = fmaf(s_cur[e >> 4][e & 15], sl2, -mc);
      pin(arg[e]);
    }
  };
  auto stage_exp = [&](int i) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = i * PER + u;
      ex[e] = fast_exp2(arg[e]);
      pin(ex[e]);
    }
  };
  auto stage_sum = [&](int i) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = i * PER + u, g = e >> 4, r = e & 15;
      if (e & 1) {
        bf16x2 pr = {(__bf16)ex[e - 1], (__bf16)ex[e]};
        pin(pr);
        p_cur[g][r >> 3][(r & 7) - 1] = pr[0];
        p_cur[g][r >> 3][r & 7] = pr[1];
        if constexpr (BS) {
          fs += ex[e - 1] + ex[e];
          pin(fs);              // in this slot: deferred, the adds keep every exponential live
        }
      }
    }
  };

#pragma unroll
  for (int i = 0; i < LA; ++i) fetch(i);
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    if (i + LA < NM) fetch(i + LA);
    mfma(i);
    if (i % RSP == RS0) rsum.add(p_prev[(i / RSP) >> 1][(i / RSP) & 1]);
    hook(i);
    stage_arg(i);
    if (i >= 1) stage_exp(i - 1);
    if (i >= 2) stage_sum(i - 2);
    __builtin_amdgcn_sched_barrier(0);
  }
  stage_exp(NM - 1);
  stage_sum(NM - 2);
  stage_sum(NM - 1);
  if constexpr (BS) *tsum = fs;
}

// One pipelined step of the block-mass pass: the NM = 2*NK QK MFMAs of the
// next tile (alternating the two 32-key groups) with, slot by slot, an equal
// share of the exp2(s * sl2 - lse2) terms of the current tile added to acc in
// (group, element) order; hook(slot) issues the caller's tile loads.
template <int D, int KS, typename Hook>
__device__ __forceinline__ void mass_step(Hook&& hook, const u16* klane, const bf16x8 (&qf)[D / 16],
                                          const f32x16 (&s_cur)[2], f32x16 (&s_next)[2], float& acc,
                                          float sl2, float nlse2) {
  constexpr int NK = D / 16, NM = 2 * NK, LA = 2;
  bf16x8 op[NM];
  auto fetch = [&](int j) {
    const int g = j & 1, ks = j >> 1;
    op[j] = *reinterpret_cast<const bf16x8*>(klane + (32 * g * KS + 2 * ks) * 8);
  };
  auto mfma = [&](int j) {
    const int g = j & 1, ks = j >> 1;
    if (ks == 0) s_next[g] = mfma32(op[j], qf[ks], f32x16{});
    else s_next[g] = mfma32(op[j], qf[ks], s_next[g]);
  };
  // Slot j owns scores [j*PER, (j+1)*PER); as in pipelined_step, slot j forms
  // their exponent arguments, slot j+1 the exponentials and slot j+2 adds
  // them to acc (in score order), the last two shares after the MFMAs.
  constexpr int PER = 32 / NM;
  float arg[32], ex[32];
  auto stage_arg = [&](int j) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = j * PER + u;
      arg[e] = fmaf(s_cur[e >> 4][e & 15], sl2, nlse2);
      pin(arg[e]);
    }
  };
  auto stage_exp = [&](int j) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = j * PER + u;
      ex[e] = fast_exp2(arg[e]);
      pin(ex[e]);
    }
  };
  auto stage_sum = [&](int j) {
#pragma unroll
    for (int u = 0; u < PER; ++u) acc += ex[j * PER + u];
    pin(acc);
  };
#pragma unroll
  for (int i = 0; i < LA; ++i) fetch(i);
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    if (i + LA < NM) fetch(i + LA);
    mfma(i);
    hook(i);
    stage_arg(i);
    if (i >= 1) stage_exp(i - 1);
    if (i >= 2) stage_sum(i - 2);
    __builtin_amdgcn_sched_barrier(0);
  }
  stage_exp(NM - 1);
  stage_sum(NM - 2);
  stage_sum(NM - 1);
}

}  // namespace adaspa
