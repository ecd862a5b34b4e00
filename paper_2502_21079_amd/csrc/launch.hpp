// Internal launch interface between the C ABI (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace adaspa {

typedef uint16_t u16;

struct AttnParams {
  const u16* q;
  const u16* k;
  const u16* v;
  u16* o;
  float* lse;                 // may be null
  const int32_t* row_ptr;     // sparse only
  const int32_t* col_idx;     // sparse only
  int64_t col_count;          // entries readable in col_idx (sparse only)
  int batch_heads;            // B * H
  int seqlen;
  int block;                  // sparse block size
  int nkb;                    // key blocks (sparse)
  int nqt;                    // query tiles per head (set by the launcher)
  int n_wg;                   // workgroups (set by the launcher)
  float scale;
  float scale_log2;           // scale * log2(e)
  int tq0, tq1;               // sparse: text query blocks [tq0, tq1), dispatched first
  int kb_guess, n_guess;      // sparse: first text block and the text block count (-1, 0: none),
                              // whose tiles every row begins with under the text sink
  uint32_t* claim;            // 9 work-queue counters (one per XCD + a flag), or null
  int n_items;                // work items: (head, query tile) or (head, query block / pair)
  int n_static;               // sparse: items [0, n_static) run in the static order
  // Single-pass search only: log2 of each row's mass in each key block,
  // [B*H, nkb, L], and log2 e * LSE of each row, [B*H, L] (scratch), and the
  // block masses W, [B*H, nkb, nkb].
  float* ylog;
  float* ylse2;
  float* wmass;
};

struct MassParams {
  const u16* q;
  const u16* k;
  const float* lse;
  float* w;                   // [B*H, nkb, nkb]
  int batch_heads;
  int seqlen;
  int block;
  int nkb;
  int n_wg;
  float scale_log2;
  uint32_t* claim;            // 8 work-queue counters (one per XCD), or null
  int n_items;                // with claim: work items (head, query-block group)
};

constexpr int kMaxHeads = 512;
constexpr int kMaxBlocks = 8192;

struct SelectParams {
  const float* w;             // [R, nb] masses, R = B*H*nb rows
  int32_t* row_ptr;
  int32_t* col_idx;
  int32_t* head_k_out;        // may be null
  float* head_recall_out;     // may be null
  // workspace
  int32_t* ws_idx;            // [R, nb] key-block order per row
  int64_t* ws_prefix;         // [R, nb] cumulative Q32 mass in that order
  int64_t* ws_curve;          // [B*H, nb] kept(k) for k = 1..nb
  int32_t* ws_headk;          // [B*H]
  int64_t* ws_base;           // [B*H] first col_idx entry of each head
  int batch_heads;
  int heads;
  int nb;
  int text_lo, text_hi;       // text block range [lo, hi]; lo > hi when none
  int kmin;                   // smallest allowed count, max(1, #text blocks)
  int mode;                   // 0 = TOPK, 1 = COVERAGE, 2 = HIERARCHICAL
  int k_base, k_hi, k_lo;     // HIERARCHICAL: counts at s, (1+s)/2 and (3s-1)/2
  int recall_thr_bp;          // HIERARCHICAL: Recall threshold
  int64_t cap;                // Q32 cap = floor(2^62 / (nb*nb))
  int32_t head_param[kMaxHeads];  // TOPK: k_h; COVERAGE: tau_bp
};

hipError_t launch_dense(AttnParams a, int head_dim, hipStream_t st);
hipError_t launch_sparse(AttnParams a, int head_dim, hipStream_t st);
hipError_t launch_block_mass(MassParams a, int head_dim, hipStream_t st);
// Dense attention + LSE and the block masses of the same rows in one launch
// (a: the attention's arguments with a.claim the optional work-queue
// counters; m: the mass pass's, its lse unused).
hipError_t launch_fused_search(AttnParams a, MassParams m, int head_dim, hipStream_t st);
// Dense attention + LSE and the block masses of its LSE in one pass over
// Q K^T (a.ylog, a.ylse2: scratch of B*H*nkb*L and B*H*L floats; a.wmass:
// the masses), then the masses summed from the scratch.
hipError_t launch_single_pass_search(AttnParams a, int head_dim, hipStream_t st);
hipError_t launch_select(const SelectParams& p, hipStream_t st);

}  // namespace adaspa
