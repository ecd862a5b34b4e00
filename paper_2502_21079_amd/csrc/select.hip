// Per-head block selection: optimal sparse indices of Sec. 4.1 (top-k of the
// block masses), text sink and row-wise uniform counts of Sec. 4.3, and the
// per-head coverage count (smallest uniform k reaching a Recall target).
//
// Determinism: the order of candidate blocks is a strict total order on
// 64-bit keys (text flag, order-preserving bits of the fp32 mass, inverted
// index), and cumulative masses are exact 64-bit integers, so every output is
// independent of thread scheduling.
#include "common.hpp"
#include "launch.hpp"

namespace adaspa {

constexpr int SEL_NT = 256;

// Order-preserving 32-bit image of an fp32 value; -0 maps like +0 and NaN
// maps below every other value.
__device__ __forceinline__ uint32_t float_order_bits(float f) {
  uint32_t b = __float_as_uint(f);
  if (f != f) return 0u;
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ int64_t q32(float m, int64_t cap) {
  if (!(m > 0.f)) return 0;                 // NaN, zeros and negatives
  double x = (double)m * 4294967296.0;
  if (!(x < 9.0e18)) return cap;            // also +inf
  long long r = llrint(x);                  // round half to even
  return r > cap ? cap : (int64_t)r;
}

__device__ __forceinline__ bool in_text(int c, int lo, int hi) { return c >= lo && c <= hi; }

// Block-wide inclusive scan of per-thread int64 totals (SEL_NT threads).
__device__ int64_t block_exclusive_scan(int64_t v, int64_t* sh, int64_t* total) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int off = 1; off < SEL_NT; off <<= 1) {
    int64_t add = tid >= off ? sh[tid - off] : 0;
    __syncthreads();
    sh[tid] += add;
    __syncthreads();
  }
  int64_t incl = sh[tid];
  if (total) *total = sh[SEL_NT - 1];
  __syncthreads();
  return incl - v;
}

// One workgroup per (b, h, p) row: order the candidate key blocks and write
// the order and the running exact sums.  Text query rows keep everything:
// their running sum is the row total at every position.
__global__ __launch_bounds__(SEL_NT) void select_rank_kernel(SelectParams P) {
  extern __shared__ uint64_t keys[];    // next power of two >= nb entries (launch size)
  __shared__ int64_t scan[SEL_NT];
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const int nb = P.nb;
  const int p = row % nb;
  const float* w = P.w + (size_t)row * nb;
  int64_t* pref = P.ws_prefix + (size_t)row * nb;
  int32_t* ord = P.ws_idx + (size_t)row * nb;
  const int per = (nb + SEL_NT - 1) / SEL_NT;   // contiguous chunk per thread
  // The curve (B*H*nb entries, one per row) is summed with atomics by the
  // next kernel: clear it here.
  if (tid == 0) P.ws_curve[row] = 0;

  if (in_text(p, P.text_lo, P.text_hi)) {
    int64_t s = 0;
    for (int i = tid * per; i < min(nb, tid * per + per); ++i) s += q32(w[i], P.cap);
    int64_t tot;
    block_exclusive_scan(s, scan, &tot);
    for (int i = tid; i < nb; i += SEL_NT) {
      pref[i] = tot;
      ord[i] = i;
    }
    return;
  }

  int n = 1;
  while (n < nb) n <<= 1;
  for (int i = tid; i < n; i += SEL_NT) {
    uint64_t kk = 0;
    if (i < nb) {
      uint64_t tf = in_text(i, P.text_lo, P.text_hi) ? 1ull : 0ull;
      kk = (tf << 63) | ((uint64_t)float_order_bits(w[i]) << 31) | (uint64_t)(0x7FFFFFFF - i);
    }
    keys[i] = kk;
  }
  __syncthreads();
  // Bitonic sort, descending.  Each stage visits its n / 2 compare-exchange
  // pairs (i, i + j) directly: i has bit j clear.
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int pr = tid; pr < (n >> 1); pr += SEL_NT) {
        const int i = ((pr & ~(j - 1)) << 1) | (pr & (j - 1));
        const int ixj = i + j;
        uint64_t x = keys[i], y = keys[ixj];
        bool desc = (i & k) == 0;
        if (desc ? (x < y) : (x > y)) {
          keys[i] = y;
          keys[ixj] = x;
        }
      }
      __syncthreads();
    }
  }
  // Running exact sums in sorted order (thread chunks are contiguous): each
  // thread sums its chunk, the chunk offsets come from a block scan, and a
  // second pass over the chunk writes the running sums.
  int64_t s = 0;
  for (int u = 0; u < per; ++u) {
    int i = tid * per + u;
    if (i < nb) {
      int idx = 0x7FFFFFFF - (int)(keys[i] & 0x7FFFFFFFull);
      ord[i] = idx;
      s += q32(w[idx], P.cap);
    }
  }
  int64_t run = block_exclusive_scan(s, scan, nullptr);
  for (int u = 0; u < per; ++u) {
    int i = tid * per + u;
    if (i < nb) {
      int idx = 0x7FFFFFFF - (int)(keys[i] & 0x7FFFFFFFull);
      run += q32(w[idx], P.cap);
      pref[i] = run;
    }
  }
}

// kept(k) of each head for k = 1..nb: sum over the head's rows.  Workgroup
// (x, bh, z) sums rows [z nb / CURVE_SPLIT, (z + 1) nb / CURVE_SPLIT) and adds
// its partial sums to the curve with 64-bit integer atomics (exact, so the
// result does not depend on their order).
constexpr int CURVE_SPLIT = 8;
__global__ __launch_bounds__(SEL_NT) void select_curve_kernel(SelectParams P) {
  const int bh = blockIdx.y;
  const int k1 = blockIdx.x * SEL_NT + threadIdx.x;
  const int nb = P.nb;
  if (k1 >= nb) return;
  const int p0 = (int)((int64_t)blockIdx.z * nb / CURVE_SPLIT);
  const int p1 = (int)((int64_t)(blockIdx.z + 1) * nb / CURVE_SPLIT);
  const int64_t* base = P.ws_prefix + (size_t)bh * nb * nb + k1;
  int64_t s = 0;
  for (int p = p0; p < p1; ++p) s += base[(size_t)p * nb];
  if (p1 > p0)
    atomicAdd(reinterpret_cast<unsigned long long*>(P.ws_curve + (size_t)bh * nb + k1),
              (unsigned long long)s);
}

// Per-head count, Recall and the first col_idx entry of every head.
__global__ __launch_bounds__(SEL_NT) void select_heads_kernel(SelectParams P) {
  __shared__ int64_t scan[SEL_NT];
  const int tid = threadIdx.x;
  const int nb = P.nb;
  const int n_text_rows = P.text_lo <= P.text_hi ? P.text_hi - P.text_lo + 1 : 0;
  int64_t carry = 0;
  for (int base = 0; base < P.batch_heads; base += SEL_NT) {
    const int bh = base + tid;
    int64_t nnz = 0;
    if (bh < P.batch_heads) {
      const int64_t* cv = P.ws_curve + (size_t)bh * nb;
      const int64_t total = cv[nb - 1];
      const int hh = bh % P.heads;
      int k;
      if (P.mode == 0) {
        k = P.head_param[hh];
      } else if (P.mode == 2) {
        // Recall of every head of this batch element at the base count; a
        // head with no mass has Recall 1.  Ranks compare kept/total exactly.
        const int b = bh / P.heads;
        const int kb = P.k_base;
        uint64_t ka = (uint64_t)cv[kb - 1], ta = (uint64_t)total;
        if (ta == 0) { ka = 1; ta = 1; }
        int n_above = 0, rank = 0;
        for (int h2 = 0; h2 < P.heads; ++h2) {
          const int64_t* c2 = P.ws_curve + (size_t)(b * P.heads + h2) * nb;
          uint64_t k2 = (uint64_t)c2[kb - 1], t2 = (uint64_t)c2[nb - 1];
          if (t2 == 0) { k2 = 1; t2 = 1; }
          n_above += ((unsigned __int128)k2 * 10000u > (unsigned __int128)t2 * (uint64_t)P.recall_thr_bp);
          const unsigned __int128 lhs = (unsigned __int128)k2 * ta, rhs = (unsigned __int128)ka * t2;
          rank += (lhs > rhs) || (lhs == rhs && h2 < hh);
        }
        const int n = n_above < P.heads / 2 ? n_above : P.heads / 2;
        k = rank < n ? P.k_hi : (rank >= P.heads - n ? P.k_lo : kb);
      } else {
        const unsigned __int128 need = (unsigned __int128)(uint64_t)total * (uint64_t)P.head_param[hh];
        int lo = P.kmin, hi = nb;   // smallest k in [lo, hi] with kept(k)*10000 >= need
        while (lo < hi) {
          int mid = (lo + hi) >> 1;
          unsigned __int128 have = (unsigned __int128)(uint64_t)cv[mid - 1] * 10000u;
          if (have >= need) hi = mid; else lo = mid + 1;
        }
        k = lo;
      }
      P.ws_headk[bh] = k;
      if (P.head_k_out) P.head_k_out[bh] = k;
      if (P.head_recall_out)
        P.head_recall_out[bh] = total == 0 ? 1.f : (float)((double)cv[k - 1] / (double)total);
      nnz = (int64_t)n_text_rows * nb + (int64_t)(nb - n_text_rows) * k;
    }
    int64_t tot;
    int64_t ex = block_exclusive_scan(nnz, scan, &tot);
    if (bh < P.batch_heads) P.ws_base[bh] = carry + ex;
    carry += tot;
  }
  if (tid == 0) P.row_ptr[(size_t)P.batch_heads * nb] = (int32_t)carry;
}

// One workgroup per row: row_ptr entry and the kept indices, ascending.
__global__ __launch_bounds__(SEL_NT) void select_emit_kernel(SelectParams P) {
  __shared__ uint8_t mark[kMaxBlocks];
  __shared__ int64_t scan[SEL_NT];
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const int nb = P.nb;
  const int bh = row / nb, p = row % nb;
  const int k = P.ws_headk[bh];
  const bool has_text = P.text_lo <= P.text_hi;
  int text_before = 0;
  if (has_text) {
    int hi = min(p, P.text_hi + 1);
    text_before = hi > P.text_lo ? hi - P.text_lo : 0;
  }
  const int64_t start = P.ws_base[bh] + (int64_t)text_before * nb + (int64_t)(p - text_before) * k;
  if (tid == 0) P.row_ptr[row] = (int32_t)start;
  int32_t* out = P.col_idx + start;
  if (in_text(p, P.text_lo, P.text_hi)) {
    for (int i = tid; i < nb; i += SEL_NT) out[i] = i;
    return;
  }
  for (int i = tid; i < nb; i += SEL_NT) mark[i] = 0;
  __syncthreads();
  const int32_t* ord = P.ws_idx + (size_t)row * nb;
  for (int i = tid; i < k; i += SEL_NT) mark[ord[i]] = 1;
  __syncthreads();
  const int per = (nb + SEL_NT - 1) / SEL_NT;
  int cnt = 0;
  for (int u = 0; u < per; ++u) {
    int i = tid * per + u;
    if (i < nb) cnt += mark[i];
  }
  int64_t pos = block_exclusive_scan(cnt, scan, nullptr);
  for (int u = 0; u < per; ++u) {
    int i = tid * per + u;
    if (i < nb && mark[i]) out[pos++] = i;
  }
}

hipError_t launch_select(const SelectParams& P, hipStream_t st) {
  const int rows = P.batch_heads * P.nb;
  int n = 1;
  while (n < P.nb) n <<= 1;
  hipLaunchKernelGGL(select_rank_kernel, dim3(rows), dim3(SEL_NT), (size_t)n * sizeof(uint64_t), st, P);
  hipLaunchKernelGGL(select_curve_kernel, dim3((P.nb + SEL_NT - 1) / SEL_NT, P.batch_heads, CURVE_SPLIT),
                     dim3(SEL_NT), 0, st, P);
  hipLaunchKernelGGL(select_heads_kernel, dim3(1), dim3(SEL_NT), 0, st, P);
  hipLaunchKernelGGL(select_emit_kernel, dim3(rows), dim3(SEL_NT), 0, st, P);
  return hipGetLastError();
}

}  // namespace adaspa
