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
// Online softmax.  The reference max of a row moves only when a tile's max
// exceeds it by more than 2^8 in the exp2 domain (checked per 32 rows), so the
// rescale of the output accumulator is skipped for almost every tile; the
// final normalisation uses the same reference, so the result is unchanged.
#pragma once

#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace adaspa {

constexpr int KT = 64;          // keys per tile
constexpr float kRescaleLog2 = 8.f;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
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

// Loads of one full K tile spread over a step (the block-mass pass).
template <int D, int NW>
struct KLoader {
  using K = TileDMA<D, NW, 1>;
  static constexpr int PW = (K::NINST + NW - 1) / NW;
  uint32_t rel[PW];

  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int i = j * NW + wave;
      rel[j] = i < K::NINST ? K::rel_offset(i, lane) : 0u;
    }
  }
  __device__ __forceinline__ void k(__amdgpu_buffer_rsrc_t r, u16* dst, uint32_t tile_byte, int j,
                                    int wave) const {
    const int i = j * NW + wave;
    if (i < K::NINST) K::issue_full(r, dst, tile_byte, i, rel[j]);
  }
};


// Loads of one full K tile and one full V tile spread over a step.  Wave w
// owns instructions i = j * NW + w of each tile; the two 16-bit in-tile
// offsets of instruction j are kept packed in one register (K low, V high).
template <int D, int NW>
struct KVLoader {
  using K = TileDMA<D, NW, 1>;
  using V = TileDMA<D, NW, 2>;
  static constexpr int PWK = (K::NINST + NW - 1) / NW;
  static constexpr int PWV = (V::NINST + NW - 1) / NW;
  static constexpr int PW = PWK > PWV ? PWK : PWV;
  static_assert(KT * D * 2 <= 65536, "in-tile offsets must fit in 16 bits");
  uint32_t rel[PW];

  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int i = j * NW + wave;
      const uint32_t k = i < K::NINST ? K::rel_offset(i, lane) : 0u;
      const uint32_t v = i < V::NINST ? V::rel_offset(i, lane) : 0u;
      rel[j] = k | (v << 16);
    }
  }
  __device__ __forceinline__ void k(__amdgpu_buffer_rsrc_t r, u16* dst, uint32_t tile_byte, int j,
                                    int wave) const {
    const int i = j * NW + wave;
    if (j < PWK && i < K::NINST) K::issue_full(r, dst, tile_byte, i, rel[j] & 0xFFFFu);
  }
  __device__ __forceinline__ void v(__amdgpu_buffer_rsrc_t r, u16* dst, uint32_t tile_byte, int j,
                                    int wave) const {
    const int i = j * NW + wave;
    if (j < PWV && i < V::NINST) V::issue_full(r, dst, tile_byte, i, rel[j] >> 16);
  }
};


// Maximum without the sNaN canonicalisation that fmaxf needs in IEEE mode
// (a NaN score propagates, which is fine: the row is then NaN either way).
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Keeps the computation of v at this point of the instruction stream: the
// empty volatile asm is ordered with the scheduling fences around it, so the
// compiler can neither sink the work that produces v past them (out of the
// MFMA slot it was placed in) nor hoist it.
__device__ __forceinline__ void pin(float& v) { asm volatile("" : "+v"(v)); }

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

// S^T tile for two groups of 32 keys: lane (hw, c32) gets keys
// 32g + 8(e/4) + 4hw + e%4 of query c32 in s[g][e].
template <int D, int S>
__device__ __forceinline__ void qk_tile(const u16* sK, const bf16x8 (&qf)[D / 16], int c32, int hw,
                                        f32x16 (&s)[2]) {
  const u16* base = sK + (c32 * S + hw) * 8;
#pragma unroll
  for (int g = 0; g < 2; ++g) {
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

// Online softmax of one S^T tile (log2 domain).  The reference max m moves
// only when some row of the wave exceeds it by more than kRescaleLog2; then
// alpha = exp2((m_old - m_new) * sl2) rescales the running sum here and the
// output accumulator later (moved tells the caller).  P is returned in bf16
// and the running sum adds exactly those rounded values, so numerator and
// denominator use the same weights.
__device__ __forceinline__ void softmax_tile(const f32x16 (&s)[2], float& m, float& lsum, float thr,
                                             float sl2, bf16x8 (&pb)[2][2], float& alpha,
                                             bool& moved) {
  float mt = -INFINITY;
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int e = 0; e < 16; e += 2) mt = vmax(mt, vmax(s[g][e], s[g][e + 1]));
  {
    float lo, hi;
    half_pair(mt, lo, hi);
    mt = vmax(lo, hi);
  }
  moved = __any(mt > m + thr);
  const float mnew = moved ? fmaxf(m, mt) : m;
  alpha = (mnew == -INFINITY) ? 1.f : fast_exp2((m - mnew) * sl2);
  lsum *= alpha;
  m = mnew;
  const float mc = (m == -INFINITY) ? 0.f : m * sl2;
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int e = 0; e < 16; ++e) pb[g][e >> 3][e & 7] = (__bf16)fast_exp2(fmaf(s[g][e], sl2, -mc));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x2 pr = {pb[g][s2][2 * j], pb[g][s2][2 * j + 1]};
        lsum = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, lsum, false);
      }
}

// O^T += V^T P^T for one tile.  MFMA step (g, s2) covers keys
// 32g + 16s2 + 8u + 4hw + j; lane (hw, e) supplies key index 8*(e/4) + 4*hw +
// e%4 of the step.  In each 16-lane group, lane j names row r0 + j/4 and 4
// elements at column d*32 + 16*(grp&1) + 4*(j%4); vlane is that lane's base.
template <int ND, int VS>
__device__ __forceinline__ void pv_tile(const u16* vlane, const bf16x8 (&pb)[2][2], f32x16 (&o)[ND]) {
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int g = 0; g < 2; ++g)
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

// One pipelined step, scheduled by hand: NM = 2*NK + 4*ND MFMA slots that
// alternate a QK MFMA (scores of the next tile) and a PV MFMA (output update
// of the previous tile).  The QK MFMAs alternate between the two 32-key score
// groups and the PV MFMAs rotate over the ND output blocks, so two MFMAs into
// the same accumulator are 4 (QK) or 2*ND (PV) slots apart and one wave alone
// keeps the matrix pipe busy; each accumulator still sums in the same order.  Each slot first issues the LDS operand reads of the
// slot LA places ahead, then its MFMA, then hook(slot) (the caller's tile
// loads, spread over the step so the load path never stalls the wave for
// long), then a fixed slice of the softmax of the current tile; a scheduling
// fence closes the slot, so the matrix pipe and the VALU work side by side
// within the wave.
template <int D, int KS, int VS, typename Hook>
__device__ __forceinline__ void pipelined_step(Hook&& hook, const u16* klane, const u16* vlane,
                                               const bf16x8 (&qf)[D / 16], const f32x16 (&s_cur)[2],
                                               const bf16x8 (&p_prev)[2][2], f32x16 (&s_next)[2],
                                               bf16x8 (&p_cur)[2][2], f32x16 (&o)[D / 32], float& m,
                                               float& lsum, float thr, float sl2, float& alpha,
                                               bool& moved) {
  constexpr int NK = D / 16, ND = D / 32;
  constexpr int NQK = 2 * NK, NPV = 4 * ND;
  static_assert(NQK == NPV, "QK and PV slots alternate");
  constexpr int NM = NQK + NPV;
  constexpr int LA = 2;                       // operand lookahead, in slots
  constexpr int P1_END = NM / 4;              // max reduction in slots [0, P1_END)
  constexpr int SHFL = P1_END;                // cross-half max exchange
  constexpr int MC = P1_END + 2;              // reference update
  constexpr int P2 = MC + 1;                  // exponentials in slots [P2, NM)

  bf16x8 op[NM];
  auto fetch = [&](int i) {
    const int j = i >> 1;
    if ((i & 1) == 0) {       // QK j: g = j % 2, ks = j / 2
      const int g = j & 1, ks = j >> 1;
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
      const int g = j & 1, ks = j >> 1;
      if (ks == 0) s_next[g] = mfma32(op[i], qf[ks], f32x16{});
      else s_next[g] = mfma32(op[i], qf[ks], s_next[g]);
    } else {
      const int d = j % ND, g = (j / ND) >> 1, s2 = (j / ND) & 1;
      o[d] = mfma32(op[i], p_prev[g][s2], o[d]);
    }
  };

  float mt = -INFINITY, mtl = -INFINITY, mth = -INFINITY, mc = 0.f;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  auto valu = [&](int i) {
    if (i < P1_END) {
      // 16 max3 over the 32 scores, spread over the first P1_END slots
      constexpr int PER = 16 / P1_END;
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int q = i * PER + u;          // pair index 0..15
        const int g = q >> 3, e = (q & 7) * 2;
        mt = vmax(mt, vmax(s_cur[g][e], s_cur[g][e + 1]));
      }
      pin(mt);
    } else if (i == SHFL) {
      half_pair(mt, mtl, mth);
    } else if (i == MC) {
      mt = vmax(mtl, mth);
      moved = __any(mt > m + thr);
      const float mnew = moved ? fmaxf(m, mt) : m;
      alpha = (mnew == -INFINITY) ? 1.f : fast_exp2((m - mnew) * sl2);
      lsum *= alpha;
      m = mnew;
      mc = (m == -INFINITY) ? 0.f : m * sl2;
      pin(mc);
    } else if (i >= P2) {
      // 32 exponentials in groups of 4 (one bf16x4 quarter of p_cur)
      constexpr int NQ = 8;                   // quarters of 4 elements
      const int k = i - P2;                   // 0 .. NM - P2 - 1
      const int q0 = k * NQ / (NM - P2), q1 = (k + 1) * NQ / (NM - P2);
#pragma unroll
      for (int q = q0; q < q1; ++q) {         // quarter q: g = q/4, elements 4*(q%4)..+3
        const int g = q >> 2, e0 = (q & 3) * 4;
#pragma unroll
        for (int e = e0; e < e0 + 4; ++e)
          p_cur[g][e >> 3][e & 7] = (__bf16)fast_exp2(fmaf(s_cur[g][e], sl2, -mc));
#pragma unroll
        for (int e = e0; e < e0 + 4; e += 2) {
          const bf16x2 pr = {p_cur[g][e >> 3][e & 7], p_cur[g][e >> 3][(e & 7) + 1]};
          lsum = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, lsum, false);
        }
      }
      pin(lsum);
    }
  };

#pragma unroll
  for (int i = 0; i < LA; ++i) fetch(i);
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    if (i + LA < NM) fetch(i + LA);
    mfma(i);
    hook(i);
    valu(i);
    __builtin_amdgcn_sched_barrier(0);
  }
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
  auto valu = [&](int j) {
    const int e0 = j * 32 / NM, e1 = (j + 1) * 32 / NM;
#pragma unroll
    for (int e = e0; e < e1; ++e) acc += fast_exp2(fmaf(s_cur[e >> 4][e & 15], sl2, nlse2));
    pin(acc);
  };
#pragma unroll
  for (int i = 0; i < LA; ++i) fetch(i);
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    if (i + LA < NM) fetch(i + LA);
    mfma(i);
    hook(i);
    valu(i);
    __builtin_amdgcn_sched_barrier(0);
  }
}

}  // namespace adaspa
