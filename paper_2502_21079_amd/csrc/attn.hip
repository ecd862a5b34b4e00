// Dense and block-sparse flash attention forward (with LSE) and the block
// attention-mass search pass, for gfx950.
//
// Orientation.  Every wave owns 32 query rows.  Scores are formed transposed,
// S^T[key][query] = K Q^T, with K as the MFMA A operand (read from LDS) and the
// wave's Q fragment as the B operand (kept in registers for the whole loop).
// In the 32x32 accumulator each lane then holds 16 keys of ONE query, so the
// softmax row statistics are lane-local plus one exchange between the two
// half-waves.  The probabilities P^T are already laid out as the B operand of
// the second product O^T[d][query] += V^T P^T, once the 16 keys of each MFMA
// step are ordered to match the accumulator rows; the V^T operand is read from
// a row-major V tile with the LDS transpose read.
#include "common.hpp"
#include "launch.hpp"

namespace adaspa {

constexpr int KT = 64;    // keys per tile
constexpr int PAD = 8;    // bf16 padding per LDS row (16 bytes)

template <int D, int NT>
struct TileIO {
  static constexpr int LDR = D + PAD;             // LDS row stride in elements
  static constexpr int CPR = D / 8;               // 16-byte chunks per row
  static constexpr int CH = KT * CPR / NT;        // chunks per thread per tile
  static_assert(KT * CPR % NT == 0, "tile chunks must divide evenly");

  // Global -> registers: rows [kbase, kbase + KT) of a [L, D] matrix; rows at
  // or beyond L read as zero.
  __device__ __forceinline__ static void load(const u16* __restrict__ src, int kbase, int L,
                                              int tid, uint4 (&r)[CH]) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      int idx = tid + c * NT;
      int row = idx / CPR, ch = idx % CPR;
      int key = kbase + row;
      if (key < L)
        r[c] = *reinterpret_cast<const uint4*>(src + (size_t)key * D + ch * 8);
      else
        r[c] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ static void store(u16* dst, int tid, const uint4 (&r)[CH]) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      int idx = tid + c * NT;
      int row = idx / CPR, ch = idx % CPR;
      *reinterpret_cast<uint4*>(dst + row * LDR + ch * 8) = r[c];
    }
  }
};

// Key tiles of one workgroup: every tile of the sequence (dense), or the
// sub-tiles of the key blocks listed in its CSR row (sparse).
template <bool SPARSE>
struct TileList {
  int n = 0;           // number of tiles
  int start = 0;       // CSR start (sparse)
  int sub = 1;         // tiles per key block (sparse)
  int block = 0, nkb = 0, L = 0;
  const int32_t* cols = nullptr;

  // Key position of tile t, or -1 when the tile holds no valid key.
  __device__ __forceinline__ int kbase(int t) const {
    if (!SPARSE) return t * KT;
    int c = cols[start + t / sub];
    if (c < 0 || c >= nkb) return -1;
    int kb = c * block + (t % sub) * KT;
    return kb < L ? kb : -1;
  }
};

// ---------------------------------------------------------------------------
// Flash attention forward (dense and block-sparse share this body).
// ---------------------------------------------------------------------------
template <int D, int NW, bool SPARSE>
__global__ __launch_bounds__(64 * NW, 2) void attn_fwd_kernel(AttnParams a) {
  constexpr int NT = 64 * NW;
  using IO = TileIO<D, NT>;
  constexpr int LDR = IO::LDR;
  constexpr int ND = D / 32;   // 32-wide output column blocks
  constexpr int NK = D / 16;   // MFMA k-steps over the head dimension
  __shared__ __attribute__((aligned(16))) u16 sK[KT * LDR];
  __shared__ __attribute__((aligned(16))) u16 sV[KT * LDR];

  const int lid = xcd_remap(blockIdx.x, a.n_wg);
  const int bh = lid / a.nqt;
  const int qt = lid % a.nqt;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hw = lane >> 5, c32 = lane & 31;
  const int L = a.seqlen;
  const size_t hoff = (size_t)bh * L * D;
  const u16* __restrict__ Kh = a.k + hoff;
  const u16* __restrict__ Vh = a.v + hoff;
  const int qrow = qt * (32 * NW) + wave * 32 + c32;

  bf16x8 qf[NK];
#pragma unroll
  for (int ks = 0; ks < NK; ++ks) {
    if (qrow < L)
      qf[ks] = *reinterpret_cast<const bf16x8*>(a.q + hoff + (size_t)qrow * D + ks * 16 + hw * 8);
    else
      qf[ks] = bf16x8{};
  }

  TileList<SPARSE> tl;
  if constexpr (SPARSE) {
    const int64_t r = (int64_t)bh * a.nkb + qt;
    int64_t s = a.row_ptr[r], e = a.row_ptr[r + 1];
    s = s < 0 ? 0 : (s > a.col_count ? a.col_count : s);
    e = e < s ? s : (e > a.col_count ? a.col_count : e);
    tl.start = (int)s;
    tl.sub = a.block / KT;
    tl.n = (int)(e - s) * tl.sub;
    tl.block = a.block;
    tl.nkb = a.nkb;
    tl.L = L;
    tl.cols = a.col_idx;
  } else {
    tl.n = (L + KT - 1) / KT;
  }

  const float sl2 = a.scale_log2;
  float m = -INFINITY, l = 0.f;
  f32x16 o[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d) o[d] = f32x16{};

  uint4 rk[IO::CH], rv[IO::CH];
  int kb_next = tl.n > 0 ? tl.kbase(0) : -1;
  if (tl.n > 0) {
    IO::load(Kh, kb_next < 0 ? L : kb_next, L, tid, rk);
    IO::load(Vh, kb_next < 0 ? L : kb_next, L, tid, rv);
    IO::store(sK, tid, rk);
    IO::store(sV, tid, rv);
  }
  __syncthreads();

  for (int t = 0; t < tl.n; ++t) {
    const int kb = kb_next;
    if (t + 1 < tl.n) {
      kb_next = tl.kbase(t + 1);
      IO::load(Kh, kb_next < 0 ? L : kb_next, L, tid, rk);
      IO::load(Vh, kb_next < 0 ? L : kb_next, L, tid, rv);
    }

    // S^T = K Q^T for two groups of 32 keys.
    f32x16 s[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      s[g] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < NK; ++ks) {
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(sK + (32 * g + c32) * LDR + ks * 16 + hw * 8);
        s[g] = mfma32(kf, qf[ks], s[g]);
      }
    }
    const int kvalid = kb < 0 ? 0 : L - kb;
    if (kvalid < KT) {
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          int key = 32 * g + 8 * (e >> 2) + 4 * hw + (e & 3);
          if (key >= kvalid) s[g][e] = -INFINITY;
        }
    }

    // Online softmax (log2 domain).
    float mt = -INFINITY;
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int e = 0; e < 16; ++e) mt = fmaxf(mt, s[g][e]);
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float mnew = fmaxf(m, mt);
    const float mc = (mnew == -INFINITY) ? 0.f : mnew * sl2;
    const float alpha = fast_exp2(m * sl2 - mc);
    float rs = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float p = fast_exp2(fmaf(s[g][e], sl2, -mc));
        rs += p;
        pb[g][e >> 3][e & 7] = (__bf16)p;
      }
    l = fmaf(l, alpha, rs);
    m = mnew;
#pragma unroll
    for (int d = 0; d < ND; ++d)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[d][e] *= alpha;

    // O^T += V^T P^T.  MFMA step (g, s2) covers keys 32g + 16s2 + 8u + 4hw + j
    // (u, j in 0..1, 0..3); lane (hw, e) supplies key index 8*(e/4) + 4*hw + e%4.
    const int gi = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int d = 0; d < ND; ++d) {
      const int dcol = d * 32 + 16 * (grp & 1) + 4 * (gi & 3);
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const u16* p0 = sV + (32 * g + 16 * s2 + 4 * hw + (gi >> 2)) * LDR + dcol;
          s16x4 lo = lds_read_tr16(p0);
          s16x4 hi = lds_read_tr16(p0 + 8 * LDR);
          bf16x8 vf;
          __builtin_memcpy(&vf, &lo, 8);
          __builtin_memcpy(reinterpret_cast<char*>(&vf) + 8, &hi, 8);
          o[d] = mfma32(vf, pb[g][s2], o[d]);
        }
    }

    __syncthreads();
    if (t + 1 < tl.n) {
      IO::store(sK, tid, rk);
      IO::store(sV, tid, rv);
    }
    __syncthreads();
  }

  // Normalise and store.
  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (qrow < L) {
    u16* orow = a.o + hoff + (size_t)qrow * D;
#pragma unroll
    for (int d = 0; d < ND; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (__bf16)(o[d][4 * i + j] * inv);
        *reinterpret_cast<bf16x4*>(orow + d * 32 + 8 * i + 4 * hw) = w;
      }
    if (hw == 0 && a.lse != nullptr)
      a.lse[(size_t)bh * L + qrow] = lt > 0.f ? fmaf(m, a.scale, logf(lt)) : -INFINITY;
  }
}

// ---------------------------------------------------------------------------
// Block attention mass: W[p][c] = sum_{i in p, j in c} exp(scale*q_i.k_j - LSE_i)
// ---------------------------------------------------------------------------
template <int D, int NW>
__global__ __launch_bounds__(64 * NW, 2) void block_mass_kernel(MassParams a) {
  constexpr int NT = 64 * NW;
  using IO = TileIO<D, NT>;
  constexpr int LDR = IO::LDR;
  constexpr int NK = D / 16;
  __shared__ __attribute__((aligned(16))) u16 sK[KT * LDR];
  __shared__ float sRed[NW];        // per-wave sums of the block just finished

  const int lid = xcd_remap(blockIdx.x, a.n_wg);
  const int bh = lid / a.nkb;
  const int p = lid % a.nkb;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hw = lane >> 5, c32 = lane & 31;
  const int L = a.seqlen;
  const size_t hoff = (size_t)bh * L * D;
  const u16* __restrict__ Kh = a.k + hoff;
  const int qrow = p * a.block + wave * 32 + c32;   // block = 32 * NW
  const bool qvalid = qrow < L;

  bf16x8 qf[NK];
#pragma unroll
  for (int ks = 0; ks < NK; ++ks) {
    if (qvalid)
      qf[ks] = *reinterpret_cast<const bf16x8*>(a.q + hoff + (size_t)qrow * D + ks * 16 + hw * 8);
    else
      qf[ks] = bf16x8{};
  }
  const float lse2 = qvalid ? a.lse[(size_t)bh * L + qrow] * kLog2e : INFINITY;
  const float sl2 = a.scale_log2;
  const int sub = a.block / KT;
  const int ntile = a.nkb * sub;

  uint4 rk[IO::CH];
  IO::load(Kh, 0, L, tid, rk);
  IO::store(sK, tid, rk);
  __syncthreads();

  float* wrow = a.w + ((size_t)bh * a.nkb + p) * a.nkb;
  float acc = 0.f;
  for (int t = 0; t < ntile; ++t) {
    const int kb = t * KT;
    if (t + 1 < ntile) IO::load(Kh, kb + KT, L, tid, rk);
    f32x16 s[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      s[g] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < NK; ++ks) {
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(sK + (32 * g + c32) * LDR + ks * 16 + hw * 8);
        s[g] = mfma32(kf, qf[ks], s[g]);
      }
    }
    const int kvalid = L - kb;
    if (kvalid < KT) {
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          int key = 32 * g + 8 * (e >> 2) + 4 * hw + (e & 3);
          if (key >= kvalid) s[g][e] = -INFINITY;
        }
    }
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc += fast_exp2(fmaf(s[g][e], sl2, -lse2));

    const bool block_end = (t + 1) % sub == 0;
    if (block_end) {
      float w = wave_sum(acc);
      if (lane == 0) sRed[wave] = w;
      acc = 0.f;
    }
    __syncthreads();
    // Waves are combined in a fixed order, so the result is deterministic.
    if (block_end && tid == 0) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += sRed[w];
      wrow[t / sub] = v;
    }
    if (t + 1 < ntile) IO::store(sK, tid, rk);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
template <int D, int NW, bool SPARSE>
static hipError_t launch_attn(const AttnParams& a, hipStream_t st) {
  hipLaunchKernelGGL((attn_fwd_kernel<D, NW, SPARSE>), dim3(a.n_wg), dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_dense(AttnParams a, int D, hipStream_t st) {
  // 128 query rows per workgroup.
  a.nqt = (a.seqlen + 127) / 128;
  a.n_wg = a.nqt * a.batch_heads;
  if (D == 64) return launch_attn<64, 4, false>(a, st);
  return launch_attn<128, 4, false>(a, st);
}

hipError_t launch_sparse(AttnParams a, int D, hipStream_t st) {
  // One workgroup per query block (block / 32 waves).
  a.nqt = a.nkb;
  a.n_wg = a.nkb * a.batch_heads;
  if (a.block == 64) {
    if (D == 64) return launch_attn<64, 2, true>(a, st);
    return launch_attn<128, 2, true>(a, st);
  }
  if (D == 64) return launch_attn<64, 4, true>(a, st);
  return launch_attn<128, 4, true>(a, st);
}

template <int D, int NW>
static hipError_t launch_mass_t(const MassParams& a, hipStream_t st) {
  hipLaunchKernelGGL((block_mass_kernel<D, NW>), dim3(a.n_wg), dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_block_mass(MassParams a, int D, hipStream_t st) {
  a.n_wg = a.nkb * a.batch_heads;
  if (a.block == 64) {
    if (D == 64) return launch_mass_t<64, 2>(a, st);
    return launch_mass_t<128, 2>(a, st);
  }
  if (D == 64) return launch_mass_t<64, 4>(a, st);
  return launch_mass_t<128, 4>(a, st);
}

}  // namespace adaspa
