// C ABI of libadaspa: argument validation on the host, then asynchronous
// launches on the caller's stream.  No device memory is allocated here.
#include <math.h>
#include <string.h>

#include <mutex>

#pragma GCC visibility push(default)
#include "adaspa.h"
#pragma GCC visibility pop
#include "launch.hpp"

using namespace adaspa;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int num_blocks(const adaspa_problem* p) { return (p->seqlen + p->block - 1) / p->block; }

// Common shape checks; returns ADASPA_OK or the status to report.
adaspa_status check_problem(const adaspa_problem* p) {
  if (!p) return ADASPA_ERR_INVALID_ARG;
  if (p->batch < 1 || p->heads < 1 || p->seqlen < 1) return ADASPA_ERR_INVALID_ARG;
  if (p->text_start < 0 || p->text_len < 0 || p->text_start > p->seqlen ||
      p->text_len > p->seqlen - p->text_start)
    return ADASPA_ERR_INVALID_ARG;
  if (!(isfinite(p->softmax_scale))) return ADASPA_ERR_INVALID_ARG;
  if (p->head_dim != 64 && p->head_dim != 128) return ADASPA_ERR_UNSUPPORTED;
  if (p->block != 64 && p->block != 128) return ADASPA_ERR_UNSUPPORTED;
  // Per-head byte sizes stay below 2^31, so every in-kernel byte offset (the
  // out-of-range offset of a skipped slot included) fits in 32 bits.
  if ((int64_t)p->seqlen * p->head_dim >= ((int64_t)1 << 30)) return ADASPA_ERR_UNSUPPORTED;
  if ((int64_t)p->batch * p->heads >= 65536) return ADASPA_ERR_UNSUPPORTED;
  return ADASPA_OK;
}

float scale_of(const adaspa_problem* p) {
  return p->softmax_scale > 0.f ? p->softmax_scale : 1.0f / sqrtf((float)p->head_dim);
}

void text_block_range(const adaspa_problem* p, bool sink, int* lo, int* hi) {
  if (!sink || p->text_len <= 0) {
    *lo = 1;
    *hi = 0;
    return;
  }
  *lo = p->text_start / p->block;
  *hi = (p->text_start + p->text_len - 1) / p->block;
}

adaspa_status check_select(const adaspa_problem* p, const adaspa_select* s) {
  if (!s) return ADASPA_ERR_INVALID_ARG;
  if (s->mode != ADASPA_SELECT_TOPK && s->mode != ADASPA_SELECT_COVERAGE &&
      s->mode != ADASPA_SELECT_HIERARCHICAL)
    return ADASPA_ERR_UNSUPPORTED;
  if (s->flags & ~(ADASPA_F_TEXT_SINK | ADASPA_F_SCORES_GIVEN)) return ADASPA_ERR_INVALID_ARG;
  if (p->heads > kMaxHeads) return ADASPA_ERR_UNSUPPORTED;
  if (num_blocks(p) > kMaxBlocks) return ADASPA_ERR_UNSUPPORTED;
  if (s->mode == ADASPA_SELECT_HIERARCHICAL) {
    if (s->base_sparsity_bp < 0 || s->base_sparsity_bp > 10000 || s->recall_threshold_bp < 0 ||
        s->recall_threshold_bp > 10000)
      return ADASPA_ERR_INVALID_ARG;
  } else {
    if (!s->head_param_bp) return ADASPA_ERR_INVALID_ARG;
    for (int h = 0; h < p->heads; ++h)
      if (s->head_param_bp[h] < 0 || s->head_param_bp[h] > 10000) return ADASPA_ERR_INVALID_ARG;
  }
  // Entries of col_idx / row_ptr are int32.
  int64_t nb = num_blocks(p);
  if ((int64_t)p->batch * p->heads * nb * nb >= ((int64_t)1 << 31)) return ADASPA_ERR_UNSUPPORTED;
  return ADASPA_OK;
}

struct WsLayout {
  size_t idx, prefix, curve, headk, base, claim, total;
};

WsLayout workspace_layout(const adaspa_problem* p) {
  const size_t bh = (size_t)p->batch * p->heads;
  const size_t nb = (size_t)num_blocks(p);
  const size_t rows = bh * nb;
  WsLayout w;
  size_t off = 0;
  w.idx = off;    off = align_up(off + rows * nb * sizeof(int32_t));
  w.prefix = off; off = align_up(off + rows * nb * sizeof(int64_t));
  w.curve = off;  off = align_up(off + bh * nb * sizeof(int64_t));
  w.headk = off;  off = align_up(off + bh * sizeof(int32_t));
  w.base = off;   off = align_up(off + bh * sizeof(int64_t));
  w.claim = off;  off = align_up(off + 9 * sizeof(uint32_t));   // mass-pass work queues (cleared as nine)
  w.total = off;
  return w;
}

int topk_count(int keep_bp, int nb, int n_text) {
  int64_t k = ((int64_t)keep_bp * nb + 9999) / 10000;
  int kmin = n_text > 1 ? n_text : 1;
  if (k > nb) k = nb;
  if (k < kmin) k = kmin;
  return (int)k;
}

// Counts of the hierarchical mode (Sec. 4.2) at sparsity s, (1+s)/2 and
// (3s-1)/2 (at least 0), all in basis points.
void hierarchical_counts(int s_bp, int nb, int n_text, int* k_base, int* k_hi, int* k_lo) {
  const int s_hi = (10000 + s_bp) / 2;
  const int s_lo3 = 3 * s_bp - 10000;
  const int s_lo = s_lo3 > 0 ? s_lo3 / 2 : 0;
  *k_base = topk_count(10000 - s_bp, nb, n_text);
  *k_hi = topk_count(10000 - s_hi, nb, n_text);
  *k_lo = topk_count(10000 - s_lo, nb, n_text);
}

// Argument checks of block-sparse attention (both entry points).
adaspa_status check_sparse(const adaspa_problem* prob, const void* q, const void* k, const void* v,
                           const int32_t* row_ptr, const int32_t* col_idx, int64_t col_count,
                           const void* out, const float* lse_out) {
  const adaspa_status st = check_problem(prob);
  if (st != ADASPA_OK) return st;
  if (!q || !k || !v || !out || !row_ptr || (!col_idx && col_count > 0) || col_count < 0)
    return ADASPA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
      (lse_out && ((uintptr_t)lse_out & 3u)) || ((uintptr_t)row_ptr & 3u) ||
      ((uintptr_t)col_idx & 3u))
    return ADASPA_ERR_INVALID_ARG;
  // Block 64 pairs query blocks through a byte map of one row's key blocks
  // (kMaxBlocks entries); block 128 has no such limit.
  if (prob->block == 64 && num_blocks(prob) > kMaxBlocks) return ADASPA_ERR_UNSUPPORTED;
  return ADASPA_OK;
}

// Scratch of adaspa_block_sparse_attn_noalloc: the per-XCD work-queue
// counters that adaspa_block_sparse_attn otherwise takes from a caller
// workspace.  Each GPU holds its own copy of this array (at its own address)
// from the library's load until the process ends.  In host code the name is
// only a stand-in for the symbol: the device address of each GPU's copy comes
// from hipGetSymbolAddress, taken once per device with that device current,
// and only that address is ever passed to a kernel.
constexpr size_t kScratchBytes = 256;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) uint32_t scratch[kScratchBytes / sizeof(uint32_t)];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch (set up on first use).
adaspa_status scratch_of_current_device(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ADASPA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return ADASPA_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return ADASPA_OK;
}

MassParams mass_params(const adaspa_problem* prob, const void* q, const void* k, const float* lse,
                       float* block_mass) {
  MassParams m;
  memset(&m, 0, sizeof m);
  m.q = (const u16*)q;
  m.k = (const u16*)k;
  m.lse = lse;
  m.w = block_mass;
  m.batch_heads = prob->batch * prob->heads;
  m.seqlen = prob->seqlen;
  m.block = prob->block;
  m.nkb = num_blocks(prob);
  m.scale_log2 = scale_of(prob) * 1.4426950408889634f;
  return m;
}

// Selection kernels of a checked search (the masses are in block_mass).
adaspa_status enqueue_selection(const adaspa_problem* prob, const adaspa_select* sel,
                                float* block_mass, int32_t* row_ptr, int32_t* col_idx,
                                int32_t* head_k, float* head_recall, void* workspace,
                                hipStream_t s) {
  const WsLayout wl = workspace_layout(prob);
  const int nb = num_blocks(prob);
  const int bh = prob->batch * prob->heads;
  SelectParams P;
  memset(&P, 0, sizeof P);
  char* ws = (char*)workspace;
  P.w = block_mass;
  P.row_ptr = row_ptr;
  P.col_idx = col_idx;
  P.head_k_out = head_k;
  P.head_recall_out = head_recall;
  P.ws_idx = (int32_t*)(ws + wl.idx);
  P.ws_prefix = (int64_t*)(ws + wl.prefix);
  P.ws_curve = (int64_t*)(ws + wl.curve);
  P.ws_headk = (int32_t*)(ws + wl.headk);
  P.ws_base = (int64_t*)(ws + wl.base);
  P.batch_heads = bh;
  P.heads = prob->heads;
  P.nb = nb;
  text_block_range(prob, (sel->flags & ADASPA_F_TEXT_SINK) != 0, &P.text_lo, &P.text_hi);
  const int n_text = P.text_lo <= P.text_hi ? P.text_hi - P.text_lo + 1 : 0;
  P.kmin = n_text > 1 ? n_text : 1;
  P.mode = sel->mode;
  P.cap = (int64_t)((((uint64_t)1) << 62) / ((uint64_t)nb * (uint64_t)nb));
  if (sel->mode == ADASPA_SELECT_HIERARCHICAL) {
    hierarchical_counts(sel->base_sparsity_bp, nb, n_text, &P.k_base, &P.k_hi, &P.k_lo);
    P.recall_thr_bp = sel->recall_threshold_bp;
  } else {
    for (int h = 0; h < prob->heads; ++h)
      P.head_param[h] = sel->mode == ADASPA_SELECT_TOPK
                            ? topk_count(sel->head_param_bp[h], nb, n_text)
                            : sel->head_param_bp[h];
  }
  return launch_select(P, s) == hipSuccess ? ADASPA_OK : ADASPA_ERR_HIP;
}

}  // namespace


#pragma GCC visibility push(default)
extern "C" {

const char* adaspa_status_string(adaspa_status s) {
  switch (s) {
    case ADASPA_OK: return "ok";
    case ADASPA_ERR_INVALID_ARG: return "invalid argument";
    case ADASPA_ERR_UNSUPPORTED: return "unsupported shape or mode";
    case ADASPA_ERR_CAPACITY: return "col_idx capacity too small";
    case ADASPA_ERR_WORKSPACE: return "workspace missing or too small";
    case ADASPA_ERR_HIP: return "HIP launch error";
  }
  return "unknown status";
}

size_t adaspa_dense_attn_workspace(const adaspa_problem* prob) {
  if (check_problem(prob) != ADASPA_OK) return 0;
  return kAlign;   // nine 32-bit work-queue counters, padded
}

size_t adaspa_block_sparse_attn_workspace(const adaspa_problem* prob) {
  if (check_problem(prob) != ADASPA_OK) return 0;
  return kAlign;   // as for dense attention
}

adaspa_status adaspa_dense_attn_lse(const adaspa_problem* prob, const void* q, const void* k,
                                    const void* v, void* out, float* lse, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  adaspa_status st = check_problem(prob);
  if (st != ADASPA_OK) return st;
  if (!q || !k || !v || !out) return ADASPA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
      (lse && ((uintptr_t)lse & 3u)))
    return ADASPA_ERR_INVALID_ARG;
  if (workspace && (workspace_bytes < adaspa_dense_attn_workspace(prob) || !aligned16(workspace)))
    return ADASPA_ERR_WORKSPACE;
  AttnParams a;
  memset(&a, 0, sizeof a);
  a.q = (const u16*)q;
  a.k = (const u16*)k;
  a.v = (const u16*)v;
  a.o = (u16*)out;
  a.lse = lse;
  a.batch_heads = prob->batch * prob->heads;
  a.seqlen = prob->seqlen;
  a.block = prob->block;
  a.nkb = num_blocks(prob);
  a.scale = scale_of(prob);
  a.scale_log2 = a.scale * 1.4426950408889634f;
  a.claim = (uint32_t*)workspace;
  return launch_dense(a, prob->head_dim, (hipStream_t)stream) == hipSuccess ? ADASPA_OK : ADASPA_ERR_HIP;
}

size_t adaspa_block_search_workspace(const adaspa_problem* prob, const adaspa_select* sel) {
  if (check_problem(prob) != ADASPA_OK || check_select(prob, sel) != ADASPA_OK) return 0;
  return workspace_layout(prob).total;
}

int64_t adaspa_block_search_capacity(const adaspa_problem* prob, const adaspa_select* sel) {
  if (check_problem(prob) != ADASPA_OK || check_select(prob, sel) != ADASPA_OK) return -1;
  const int64_t nb = num_blocks(prob);
  const int64_t bh = (int64_t)prob->batch * prob->heads;
  if (sel->mode == ADASPA_SELECT_COVERAGE) return bh * nb * nb;
  int lo, hi;
  text_block_range(prob, (sel->flags & ADASPA_F_TEXT_SINK) != 0, &lo, &hi);
  const int n_text = lo <= hi ? hi - lo + 1 : 0;
  if (sel->mode == ADASPA_SELECT_HIERARCHICAL) {
    int kb, kh, kl;
    hierarchical_counts(sel->base_sparsity_bp, (int)nb, n_text, &kb, &kh, &kl);
    int kmax = kb > kh ? kb : kh;
    kmax = kmax > kl ? kmax : kl;
    return bh * (n_text * nb + (nb - n_text) * kmax);
  }
  int64_t total = 0;
  for (int h = 0; h < prob->heads; ++h) {
    const int k = topk_count(sel->head_param_bp[h], (int)nb, n_text);
    total += n_text * nb + (nb - n_text) * k;
  }
  return total * prob->batch;
}

adaspa_status adaspa_block_search(const adaspa_problem* prob, const void* q, const void* k,
                                  const float* lse, const adaspa_select* sel, float* block_mass,
                                  int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                  int32_t* head_k, float* head_recall, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  adaspa_status st = check_problem(prob);
  if (st != ADASPA_OK) return st;
  st = check_select(prob, sel);
  if (st != ADASPA_OK) return st;
  const bool given = (sel->flags & ADASPA_F_SCORES_GIVEN) != 0;
  if (!block_mass || !row_ptr || !col_idx) return ADASPA_ERR_INVALID_ARG;
  if (!given) {
    if (!q || !k || !lse) return ADASPA_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || ((uintptr_t)lse & 3u)) return ADASPA_ERR_INVALID_ARG;
  }
  if (((uintptr_t)block_mass & 3u) || ((uintptr_t)row_ptr & 3u) || ((uintptr_t)col_idx & 3u))
    return ADASPA_ERR_INVALID_ARG;
  const int64_t need = adaspa_block_search_capacity(prob, sel);
  if (col_capacity < need) return ADASPA_ERR_CAPACITY;
  const WsLayout wl = workspace_layout(prob);
  if (!workspace || workspace_bytes < wl.total || ((uintptr_t)workspace % kAlign))
    return ADASPA_ERR_WORKSPACE;

  hipStream_t s = (hipStream_t)stream;
  if (!given) {
    MassParams m = mass_params(prob, q, k, lse, block_mass);
    m.claim = (uint32_t*)((char*)workspace + wl.claim);
    if (launch_block_mass(m, prob->head_dim, s) != hipSuccess) return ADASPA_ERR_HIP;
  }
  return enqueue_selection(prob, sel, block_mass, row_ptr, col_idx, head_k, head_recall, workspace, s);
}

adaspa_status adaspa_fused_online_search(const adaspa_problem* prob, const void* q, const void* k,
                                         const void* v, void* out, float* lse,
                                         const adaspa_select* sel, float* block_mass,
                                         int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                         int32_t* head_k, float* head_recall, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  adaspa_status st = check_problem(prob);
  if (st != ADASPA_OK) return st;
  st = check_select(prob, sel);
  if (st != ADASPA_OK) return st;
  if (sel->flags & ADASPA_F_SCORES_GIVEN) return ADASPA_ERR_INVALID_ARG;
  if (!q || !k || !v || !out || !block_mass || !row_ptr || !col_idx) return ADASPA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
      (lse && ((uintptr_t)lse & 3u)) || ((uintptr_t)block_mass & 3u) ||
      ((uintptr_t)row_ptr & 3u) || ((uintptr_t)col_idx & 3u))
    return ADASPA_ERR_INVALID_ARG;
  const int64_t need = adaspa_block_search_capacity(prob, sel);
  if (col_capacity < need) return ADASPA_ERR_CAPACITY;
  const WsLayout wl = workspace_layout(prob);
  if (!workspace || workspace_bytes < wl.total || ((uintptr_t)workspace % kAlign))
    return ADASPA_ERR_WORKSPACE;

  hipStream_t s = (hipStream_t)stream;
  AttnParams a;
  memset(&a, 0, sizeof a);
  a.q = (const u16*)q;
  a.k = (const u16*)k;
  a.v = (const u16*)v;
  a.o = (u16*)out;
  a.lse = lse;
  a.batch_heads = prob->batch * prob->heads;
  a.seqlen = prob->seqlen;
  a.block = prob->block;
  a.nkb = num_blocks(prob);
  a.scale = scale_of(prob);
  a.scale_log2 = a.scale * 1.4426950408889634f;
  a.claim = (uint32_t*)((char*)workspace + wl.claim);
  const MassParams m = mass_params(prob, q, k, lse, block_mass);
  if (launch_fused_search(a, m, prob->head_dim, s) != hipSuccess) return ADASPA_ERR_HIP;
  return enqueue_selection(prob, sel, block_mass, row_ptr, col_idx, head_k, head_recall, workspace, s);
}

// Bytes of the single pass's scratch for heads_per_call (batch, head) pairs
// at a time: the per-row block masses and row LSEs of those pairs, after the
// search's workspace (which the selection of all heads uses).
static size_t single_pass_bytes(const adaspa_problem* prob, size_t heads_per_call) {
  return workspace_layout(prob).total +
         align_up(heads_per_call * (size_t)num_blocks(prob) * prob->seqlen * sizeof(float)) +
         align_up(heads_per_call * (size_t)prob->seqlen * sizeof(float));
}

size_t adaspa_single_pass_online_search_workspace(const adaspa_problem* prob, const adaspa_select* sel) {
  if (check_problem(prob) != ADASPA_OK || check_select(prob, sel) != ADASPA_OK) return 0;
  if (sel->flags & ADASPA_F_SCORES_GIVEN) return 0;
  return single_pass_bytes(prob, (size_t)prob->batch * prob->heads);
}

size_t adaspa_single_pass_online_search_min_workspace(const adaspa_problem* prob, const adaspa_select* sel) {
  if (check_problem(prob) != ADASPA_OK || check_select(prob, sel) != ADASPA_OK) return 0;
  if (sel->flags & ADASPA_F_SCORES_GIVEN) return 0;
  return single_pass_bytes(prob, 1);
}

adaspa_status adaspa_single_pass_online_search(const adaspa_problem* prob, const void* q, const void* k,
                                               const void* v, void* out, float* lse,
                                               const adaspa_select* sel, float* block_mass,
                                               int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                               int32_t* head_k, float* head_recall, void* workspace,
                                               size_t workspace_bytes, void* stream) {
  adaspa_status st = check_problem(prob);
  if (st != ADASPA_OK) return st;
  st = check_select(prob, sel);
  if (st != ADASPA_OK) return st;
  if (sel->flags & ADASPA_F_SCORES_GIVEN) return ADASPA_ERR_INVALID_ARG;
  if (!q || !k || !v || !out || !block_mass || !row_ptr || !col_idx) return ADASPA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
      (lse && ((uintptr_t)lse & 3u)) || ((uintptr_t)block_mass & 3u) ||
      ((uintptr_t)row_ptr & 3u) || ((uintptr_t)col_idx & 3u))
    return ADASPA_ERR_INVALID_ARG;
  const int64_t need = adaspa_block_search_capacity(prob, sel);
  if (col_capacity < need) return ADASPA_ERR_CAPACITY;
  if (!workspace || workspace_bytes < single_pass_bytes(prob, 1) || ((uintptr_t)workspace % kAlign))
    return ADASPA_ERR_WORKSPACE;
  // As many (batch, head) pairs per launch as the workspace holds: all of
  // them with adaspa_single_pass_online_search_workspace() bytes.  Each pair
  // is computed the same way whatever its group, so the results do not
  // depend on the grouping.
  const int bh_all = prob->batch * prob->heads;
  int g = bh_all;
  while (g > 1 && single_pass_bytes(prob, (size_t)g) > workspace_bytes) g = g / 2 > 1 ? g / 2 : 1;
  while (g < bh_all && single_pass_bytes(prob, (size_t)g + 1) <= workspace_bytes) ++g;

  hipStream_t s = (hipStream_t)stream;
  const WsLayout wl = workspace_layout(prob);
  const size_t L = (size_t)prob->seqlen, D = (size_t)prob->head_dim, nkb = (size_t)num_blocks(prob);
  for (int g0 = 0; g0 < bh_all; g0 += g) {
    const int gn = bh_all - g0 < g ? bh_all - g0 : g;
    AttnParams a;
    memset(&a, 0, sizeof a);
    a.q = (const u16*)q + (size_t)g0 * L * D;
    a.k = (const u16*)k + (size_t)g0 * L * D;
    a.v = (const u16*)v + (size_t)g0 * L * D;
    a.o = (u16*)out + (size_t)g0 * L * D;
    a.lse = lse ? lse + (size_t)g0 * L : nullptr;
    a.batch_heads = gn;
    a.seqlen = prob->seqlen;
    a.block = prob->block;
    a.nkb = (int)nkb;
    a.scale = scale_of(prob);
    a.scale_log2 = a.scale * 1.4426950408889634f;
    a.claim = (uint32_t*)((char*)workspace + wl.claim);
    a.ylog = (float*)((char*)workspace + wl.total);
    a.ylse2 = (float*)((char*)workspace + wl.total + align_up((size_t)gn * nkb * L * sizeof(float)));
    a.wmass = block_mass + (size_t)g0 * nkb * nkb;
    if (launch_single_pass_search(a, prob->head_dim, s) != hipSuccess) return ADASPA_ERR_HIP;
  }
  return enqueue_selection(prob, sel, block_mass, row_ptr, col_idx, head_k, head_recall, workspace, s);
}

adaspa_status adaspa_block_sparse_attn(const adaspa_problem* prob, const void* q, const void* k,
                                       const void* v, const int32_t* row_ptr,
                                       const int32_t* col_idx, int64_t col_count, void* out,
                                       float* lse_out, void* workspace, size_t workspace_bytes,
                                       void* stream) {
  const adaspa_status st = check_sparse(prob, q, k, v, row_ptr, col_idx, col_count, out, lse_out);
  if (st != ADASPA_OK) return st;
  if (workspace && (workspace_bytes < adaspa_block_sparse_attn_workspace(prob) || !aligned16(workspace)))
    return ADASPA_ERR_WORKSPACE;
  AttnParams a;
  memset(&a, 0, sizeof a);
  a.q = (const u16*)q;
  a.k = (const u16*)k;
  a.v = (const u16*)v;
  a.o = (u16*)out;
  a.lse = lse_out;
  a.row_ptr = row_ptr;
  a.col_idx = col_idx;
  a.col_count = col_count;
  a.batch_heads = prob->batch * prob->heads;
  a.seqlen = prob->seqlen;
  a.block = prob->block;
  a.nkb = num_blocks(prob);
  a.scale = scale_of(prob);
  a.scale_log2 = a.scale * 1.4426950408889634f;
  a.claim = (uint32_t*)workspace;
  // Text query blocks keep every key block under the text sink, so they are
  // the longest rows; the kernel starts them first (the result does not
  // depend on the order).
  if (prob->text_len > 0) {
    a.tq0 = prob->text_start / prob->block;
    a.tq1 = (prob->text_start + prob->text_len + prob->block - 1) / prob->block;
    if (a.tq1 - a.tq0 >= a.nkb) a.tq0 = a.tq1 = 0;    // every row is text: plain order
  }
  a.kb_guess = a.tq1 > a.tq0 ? a.tq0 : -1;
  a.n_guess = a.tq1 - a.tq0;
  return launch_sparse(a, prob->head_dim, (hipStream_t)stream) == hipSuccess ? ADASPA_OK : ADASPA_ERR_HIP;
}

adaspa_status adaspa_block_sparse_attn_noalloc(const adaspa_problem* prob, const void* q,
                                               const void* k, const void* v,
                                               const int32_t* row_ptr, const int32_t* col_idx,
                                               int64_t col_count, void* out, float* lse_out,
                                               void* stream) {
  const adaspa_status st = check_sparse(prob, q, k, v, row_ptr, col_idx, col_count, out, lse_out);
  if (st != ADASPA_OK) return st;
  // The counters need the same bytes for every problem; the check keeps the
  // limit explicit should that ever change.
  const size_t need = adaspa_block_sparse_attn_workspace(prob);
  if (need == 0 || need > kScratchBytes) return ADASPA_ERR_WORKSPACE;
  void* ws = nullptr;
  const adaspa_status ss = scratch_of_current_device(&ws);
  if (ss != ADASPA_OK) return ss;
  return adaspa_block_sparse_attn(prob, q, k, v, row_ptr, col_idx, col_count, out, lse_out, ws,
                                  kScratchBytes, stream);
}

}  // extern "C"
#pragma GCC visibility pop
