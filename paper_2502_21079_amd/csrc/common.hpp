// Shared device helpers for the gfx950 (CDNA4) kernels of the AdaSpa path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace adaspa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// C[32x32] += A[32x16] * B[16x32] on bf16 inputs, fp32 accumulate.
// Lane l supplies A[l%32][8*(l/32) + e] and B[8*(l/32) + e][l%32], e = 0..7;
// accumulator element 4*i + j of lane l is C[8*i + 4*(l/32) + j][l%32].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// LDS transpose read of 16-bit elements.  Within each group of 16 lanes, lane
// j names 4 consecutive elements R[j][0..3]; lane i receives R[i/4 + 4e][i%4]
// for e = 0..3.
__device__ __forceinline__ s16x4 lds_read_tr16(const u16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(p));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup i runs on
// XCD i % 8).  Map hardware id -> logical id so that each XCD receives one
// contiguous range of logical ids: neighbouring tiles of one head then share
// that XCD's L2.  Bijective for any n.
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int nx = 8;
  int q = n / nx, r = n % nx;
  int x = bid % nx, k = bid / nx;
  int off = x * q + (x < r ? x : r);
  return off + k;
}

// Lane l's value and lane (l ^ 32)'s value, returned as (a, b) in an order
// that depends on the half-wave: a = v[l & 31], b = v[(l & 31) + 32].  One
// v_permlane32_swap (a VALU op; no LDS round trip as with a shuffle).
__device__ __forceinline__ void half_pair(float v, float& a, float& b) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}

// Sum over the 64 lanes of a wave, returned to every lane.  DPP moves sum
// within each row of 16 lanes (no LDS round trips); the four row sums are
// then read out and added in a fixed order, so the result is deterministic.
template <int CTRL>
__device__ __forceinline__ float dpp_plus(float v) {
  const int moved = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false);
  return v + __builtin_bit_cast(float, moved);
}
// Work order of block-sparse attention.  Long rows first: the nt = ntq * nbh
// workgroups of the ntq query tiles [tq0, tq0 + ntq) of every head are
// dispatched first (hardware ids 0..nt-1, spread round-robin over the XCDs);
// in block-sparse attention the text query blocks keep every key block, so
// they are the longest rows by far, and starting them first removes the tail
// they would otherwise leave.  The other tiles follow in (chunk, head, tile)
// order, chunk c holding tiles [c*m/8, (c+1)*m/8) of every head (m tiles per
// head), and each XCD receives one contiguous range of that order: it works
// on contiguous runs of query tiles, whose neighbours keep largely the same
// key blocks (they share its L2), and on an equal share of every head (heads
// of different cost stay balanced).  Bijective for any sizes.
__device__ __forceinline__ void text_first_map(int hid, int n, int nqt, int tq0, int ntq, int& bh,
                                               int& qt) {
  const int nbh = n / nqt;
  const int nt = ntq * nbh;
  if (hid < nt) {
    bh = hid / ntq;
    qt = tq0 + hid % ntq;
    return;
  }
  auto cnt = [](int N, int y) { return N > y ? (N + 7 - y) / 8 : 0; };   // ids < N on XCD y
  const int x = hid % 8;
  int lid = cnt(hid, x) - cnt(nt, x);
  for (int y = 0; y < x; ++y) lid += cnt(n, y) - cnt(nt, y);
  const int nvq = nqt - ntq;
  int c = 0, start = 0;
  for (; c < 7; ++c) {
    const int sz = ((c + 1) * nvq) / 8 - (c * nvq) / 8;
    if (lid < start + sz * nbh) break;
    start += sz * nbh;
  }
  const int c0 = (c * nvq) / 8, sz = ((c + 1) * nvq) / 8 - c0;
  bh = (lid - start) / sz;
  const int r = c0 + (lid - start) % sz;
  qt = r < tq0 ? r : r + ntq;
}

__device__ __forceinline__ float wave_sum(float v) {
  v = dpp_plus<0xB1>(v);    // quad_perm [1,0,3,2]: pairs
  v = dpp_plus<0x4E>(v);    // quad_perm [2,3,0,1]: quads
  v = dpp_plus<0x124>(v);   // row_ror:4: two quads
  v = dpp_plus<0x128>(v);   // row_ror:8: whole row of 16
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (r0 + r1) + (r2 + r3);
}

}  // namespace adaspa
