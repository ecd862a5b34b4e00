// Dense and block-sparse flash attention forward (32 query rows per wave) and
// the block attention-mass search pass, for gfx950.
//
// Pipeline.  K/V tiles of 64 keys sit in LDS rings and are filled by direct
// global->LDS buffer loads (no register staging), issued one or two steps
// before the tiles are read, one per MFMA slot at the front of a step.  Only a
// tile that reaches past the end of the sequence pays for key masking.
#include "attn_tile.hpp"

namespace adaspa {

// Dynamic work distribution over the XCDs.  The XCDs of one chip do not run
// at the same speed (per-XCD step times differ by up to ~10% on the same
// work), so a static equal split leaves the fast ones idle at the end.  Work
// item i (in the kernel's static order) belongs to the queue of XCD i % 8, as
// the hardware's round-robin dispatch would place it; a workgroup takes the
// next item of its own XCD's queue with an atomic increment and, once that is
// empty, the next item of another queue, and exits when all are empty.  The
// grid has more workgroups than items, so a faster XCD simply runs more of
// them.  Items keep their order within a queue, so neighbouring tiles still
// share an L2.  Block-sparse attention runs the first nine tenths of its
// items in the static order and queues only the rest: on its short rows the
// claim's round trip would otherwise sit in every workgroup's prologue.
__device__ __forceinline__ int xcc_id() {
  return __builtin_amdgcn_s_getreg(20 | (0 << 6) | (3 << 11)) & 7;   // HW_REG_XCC_ID[3:0]
}

// Takes an item of [n0, n) (n0 a multiple of 8, so item n0 + y + 8j is in
// queue y), or returns -1 when every queue is empty.  With FLAG, ctr[8] is
// set once a workgroup has found all queues empty, and later workgroups
// return after reading it instead of trying all eight counters.
template <bool FLAG = false>
__device__ __forceinline__ int claim_item(uint32_t* ctr, int n0, int n) {
  if (FLAG && __atomic_load_n(&ctr[8], __ATOMIC_RELAXED) != 0u) return -1;
  const int x = xcc_id();
  for (int k = 0; k < 8; ++k) {
    const int y = (x + k) & 7;
    const int m = (n - n0 - y + 7) / 8;       // items of queue y
    const unsigned j = atomicAdd(&ctr[y], 1u);
    if ((int)j < m) return n0 + (int)j * 8 + y;
  }
  if (FLAG) atomicExch(&ctr[8], 1u);
  return -1;
}

__global__ void claim_reset_kernel(uint32_t* ctr) {
  if (threadIdx.x < 9) ctr[threadIdx.x] = 0u;
}

// ---------------------------------------------------------------------------
// Flash attention forward (dense and block-sparse share this body).
//
// Full key tiles run through a software pipeline: step t computes the scores
// of tile t+1 (QK MFMAs) and the output update of tile t-1 (PV MFMAs) while
// the VALU does the softmax of tile t.  K therefore runs one tile ahead of the
// scores and V one tile behind (the K/V rings are described below).  A tile that
// reaches past the end of the sequence (and, in a malformed sparse row, any
// out-of-range block) is done afterwards, one at a time with key masking,
// which keeps the visiting order of the dense and all-blocks sparse paths the
// same.  After the rows are stored, tail() may continue with the same rows
// (the fused search below); the attention kernels pass NoTail.
// ---------------------------------------------------------------------------
struct NoTail {
  template <typename... T>
  __device__ __forceinline__ void operator()(T&&...) const {}
};

// With BS (dense only) the body also writes, for every row and key block c,
// log2 of the row's unnormalised mass in block c plus the row's reference at
// that time, so that the block's share of the row's softmax is
// exp2(ylog - LSE * log2(e)) (the single-pass search below).
template <int D, int NW, bool SPARSE, bool BS = false, typename Tail>
__device__ __forceinline__ void attn_fwd_body(AttnParams a, Tail&& tail) {
  static_assert(!(SPARSE && BS), "block masses come from the dense pass");
  constexpr int NT = 64 * NW;
  using KDMA = TileDMA<D, NW, 1>;
  using VDMA = TileDMA<D, NW, 2>;
  constexpr int KS = KDMA::S, VS = VDMA::S;
  constexpr int ND = D / 32;   // 32-wide output column blocks
  constexpr int NK = D / 16;   // MFMA k-steps over the head dimension
  // A ring of two slots, each [K tile | V tile]; step t reads K(t+1) and
  // V(t-1) from one slot while K(t+2) and V(t) are loaded into the other,
  // and the waves meet at a barrier every step.  (Two slots measured faster
  // than four with a barrier every second step for the dense kernel.)
  using LD = KVLoader<D, NW>;
  constexpr int RING = 2;
  __shared__ __attribute__((aligned(1024))) u16 sKV[RING][LD::ELEMS];   // slots [K | V]
  const SlotPart<LD::ELEMS, 0> sK{sKV};
  const SlotPart<LD::ELEMS, LD::VOFF> sV{sKV};

  // Work mapping.  Block-sparse: the text query blocks of every head first,
  // then an equal contiguous share of every head's video query blocks per
  // XCD (text_first_map).  Dense: one contiguous range of (head, query tile)
  // items per XCD (xcd_remap), through the per-XCD queues when a workspace
  // is given.
  int bh, qt;
  if constexpr (SPARSE) {
    int item = (int)blockIdx.x;
    if (item >= a.n_static) {                // the queued tail (see claim_item)
      __shared__ int s_tail;
      if (threadIdx.x == 0) s_tail = claim_item<true>(a.claim, a.n_static, a.n_items);
      __syncthreads();
      item = s_tail;
      if (item < 0) return;
    }
    text_first_map(item, a.n_items, a.nqt, a.tq0, a.tq1 - a.tq0, bh, qt);
  } else {
    int item = (int)blockIdx.x;
    if (a.claim != nullptr) {
      __shared__ int s_item;
      if (threadIdx.x == 0) s_item = claim_item(a.claim, 0, a.n_items);
      __syncthreads();
      item = s_item;
      if (item < 0) return;                  // every item is taken
    }
    const int lid = xcd_remap(item, a.n_items);
    bh = lid / a.nqt;
    qt = lid % a.nqt;
  }
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int hw = lane >> 5, c32 = lane & 31;
  const int gi = lane & 15, grp = lane >> 4;
  const int L = a.seqlen;
  const size_t hoff = (size_t)bh * L * D;
  const uint32_t hbytes = (uint32_t)L * D * 2u;
  const __amdgpu_buffer_rsrc_t rK = make_rsrc(a.k + hoff, hbytes);
  const __amdgpu_buffer_rsrc_t rV = make_rsrc(a.v + hoff, hbytes);
  const u32x4 rKw = rsrc_words(a.k + hoff, hbytes), rVw = rsrc_words(a.v + hoff, hbytes);
  const int qrow = qt * (32 * NW) + wave * 32 + c32;
  const int voff = ((4 * hw + (gi >> 2)) * VS) * 8 + 16 * (grp & 1) + 4 * (gi & 3);
  const int klane = (c32 * KS + hw) * 8;

  // V slots hold finite values whatever a bounds-checked load leaves behind
  // (a key masked to -inf still multiplies its V row by a zero probability);
  // K rows past the sequence are masked whatever they hold.
#pragma unroll
  for (int b = 0; b < RING; ++b) zero_lds<VDMA::SLOTS>(sV[b], tid, NT);

  bf16x8 qf[NK];
  load_q<D>(a.q + hoff, qrow, L, hw, qf);

  // Sparse rows ordered with a text range start, under the text sink, with
  // the first text block: its first two tiles are loaded into place before
  // the row's indices are read (a guess, checked below), which takes the
  // index round trips off the path to the first tile.
  const int spec = (SPARSE && a.kb_guess >= 0) ? a.kb_guess * a.block : -1;
  if (spec >= 0) {
    KDMA::issue(rK, sK[0], spec, wave, lane);
    KDMA::issue(rK, sK[1], spec + KT, wave, lane);
  }

  // Tiles: nf full tiles through the pipeline; the rest one by one, masked.
  int nf = 0;                 // full tiles in the pipeline
  int e0 = 0, ne = 0;         // sparse: CSR entries [e0, e0 + ne)
  int skip = -1;              // sparse: entry (relative) holding the ragged block
  bool slow = false;          // sparse: malformed row, take the masked path for all
  constexpr int SUB = SPARSE ? NW / 2 : 1;   // KT-key tiles per sparse block (block = 32 * NW)
  const int sub = SUB;
  // Sparse: the row's block indices are read 64 at a time into one register
  // per lane (entry n sits in lane n % 64 of chunk n / 64) and picked out
  // with readlane; a window of two chunks moves along the row, so no index
  // load is waited for inside the main loop.
  // The loads go through a resource bounded to the row, so lanes past its end
  // read 0 without a branch and each chunk lands directly in its register.
  __amdgpu_buffer_rsrc_t rC = make_rsrc(a.col_idx, 0u);
  auto load_chunk = [&](int c) -> int {
    return __builtin_amdgcn_raw_buffer_load_b32(rC, (uint32_t)(c * 64 + lane) * 4u, 0, 0);
  };
  int c0 = 0, cid0 = 0, cid1 = 0;
  int skip_at = INT_MAX;      // sparse: pipeline entries at or past it shift by one
  int rag_sub = 0;            // sparse: full tiles of the ragged entry taken by the pipeline
  if constexpr (SPARSE) {
    const int64_t r = (int64_t)bh * a.nkb + qt;
    int64_t s = a.row_ptr[r], e = a.row_ptr[r + 1];
    s = s < 0 ? 0 : (s > a.col_count ? a.col_count : s);
    e = e < s ? s : (e > a.col_count ? a.col_count : e);
    e0 = (int)s;
    ne = (int)(e - s);
    rC = make_rsrc(a.col_idx + e0, (uint32_t)ne * 4u);
    // The first two chunks are the window's; the validation scan reads them
    // from there (one memory round trip less before the first tile loads).
    cid0 = load_chunk(0);
    cid1 = load_chunk(1);
    const bool ragged = L % a.block != 0;
    for (int c = 0; c * 64 < ne; ++c) {
      const int n = c * 64 + lane;
      const int v = c == 0 ? cid0 : (c == 1 ? cid1 : load_chunk(c));
      if (__any(n < ne && (v < 0 || v >= a.nkb))) slow = true;
      const unsigned long long rb = __ballot(n < ne && ragged && v == a.nkb - 1);
      if (skip < 0 && rb != 0ull) skip = c * 64 + __builtin_ctzll(rb);
    }
    // A ragged block that ends the row (the usual, ascending case) keeps its
    // full tiles in the pipeline, as the dense kernel does, and only its
    // partial tile is masked; elsewhere it is left out whole.
    if (!slow && skip >= 0 && skip == ne - 1) rag_sub = (L - (a.nkb - 1) * a.block) / KT;
    nf = slow ? 0 : (ne - (skip >= 0 ? 1 : 0)) * SUB + rag_sub;
    skip_at = (skip >= 0 && skip != ne - 1) ? skip : INT_MAX;
  } else {
    nf = L / KT;
  }
  auto entry = [&](int t) -> int {     // CSR entry of pipeline tile t
    const int i = t / SUB;
    return i + (i >= skip_at ? 1 : 0);
  };
  auto kbase = [&](int t) -> int {
    if constexpr (!SPARSE) {
      return t * KT;
    } else {
      const int i = entry(t);
      const int v0 = __builtin_amdgcn_readlane(cid0, i & 63);
      const int v1 = __builtin_amdgcn_readlane(cid1, i & 63);
      return ((i >> 6) == c0 ? v0 : v1) * (SUB * KT) + (t % SUB) * KT;
    }
  };

  const float sl2 = a.scale_log2;
  RowRef ref;                             // softmax reference of this lane's row
  float lsum = 0.f;                       // this lane's half of the row sum
  // BS: this lane's fp32 sum of exp2(s * sl2 - ref.mc) over the current key
  // block so far; written out (both halves of the row added) when the block
  // ends, as log2 of the sum plus ref.mc.  rowf is the same sum over the whole
  // row: the masses are normalised by it rather than by the sum of the
  // bf16-rounded weights behind the output and its LSE, whose rounding (up
  // to 2^-9 of a weight) would shift every mass of a row dominated by a few
  // keys by as much.
  float bsum = 0.f, rowf = 0.f;
  const int tsh = (BS && a.block == 128) ? 1 : 0;   // log2 of the tiles per key block
  const int tpb = 1 << tsh;
  // BS, pipelined tiles: the sum of a key block that ended at step t waits in
  // bdone and is written in the middle of step t + 1, under its MFMAs, so
  // the end of step t does not wait for that step's last additions, the
  // exchange and the logarithm.  It is relative to the reference of step t,
  // which moves again only after step t + 1's MFMAs.  cdone is its key
  // block, -1 when none waits.
  float bdone = 0.f;
  int cdone = -1;
  auto write_block = [&](float bs, int c) {
    if constexpr (BS) {
      float lo, hi;
      half_pair(bs, lo, hi);
      const float b = lo + hi;
      // Column c of this head's [nkb, L] slab: a wave-uniform base, and the
      // row as a 32-bit offset.
      float* col = a.ylog + ((size_t)bh * a.nkb + (size_t)__builtin_amdgcn_readfirstlane(c)) * (size_t)L;
      if (hw == 0 && qrow < L) col[qrow] = (b > 0.f ? __builtin_amdgcn_logf(b) : -INFINITY) + ref.mc;
    }
  };
  auto flush_block = [&](int c) {
    if constexpr (BS) {
      write_block(bsum, c);
      bsum = 0.f;
    }
  };
  auto flush_waiting = [&]() {
    if constexpr (BS) {
      if (cdone >= 0) {
        write_block(bdone, cdone);
        cdone = -1;
      }
    }
  };
  f32x16 o[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d) o[d] = f32x16{};
  // A wave whose row sums left the safe range redoes its rows on the exact
  // (masked) path; the workgroup walks the tiles together for the loads and
  // barriers, and only that wave computes.
  __shared__ int s_redo;
  if (tid == 0) s_redo = 0;
  bool redo = false;                      // this wave redoes its rows
  __syncthreads();

  if (nf > 0) {
    // Step t reads K(t+1) and V(t-1), so the first steps need K(0) and K(1)
    // in place.  A wrong guess is overwritten once this wave's guessed loads
    // have landed (each wave reloads the same pieces of the slots).
    const int kb0 = kbase(0), kb1 = nf > 1 ? kbase(1) : -1;
    if (!(spec >= 0 && kb0 == spec && (nf < 2 || kb1 == spec + KT))) {
      if (spec >= 0) wait_vmem();
      KDMA::issue(rK, sK[0], kb0, wave, lane);
      if (nf > 1) KDMA::issue(rK, sK[1], kb1, wave, lane);
    }
    wait_vmem();
    __syncthreads();
    f32x16 s_cur[2];
    qk_tile<D, KS>(sK[0], qf, c32, hw, s_cur);
    __syncthreads();            // slot 0 is refilled by step 0

    bf16x8 p_prev[2][2];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) p_prev[g][s2] = bf16x8{};
    bool pend = false;
    float pend_alpha = 1.f;
    RowSums rsum;
    rsum.init(lane);
    bool bad = false;

    LD ld;
    ld.init(wave, lane);
    const u32x4 rMw = ld.mixed_v ? rVw : rKw;     // resource of this wave's mixed entry

    // Step t reads K(t+1) and V(t-1) from slot (t+1)&1 and loads K(t+2) and
    // V(t) into slot t&1, which step t-1 read: a slot is refilled only after
    // the barrier that follows the step which read it, and a loaded tile is
    // read only after the barrier that follows its loads.  The loads take
    // the first MFMA slots of the step, one per slot.  Past the last tile the K
    // index is clamped to the last one (an in-range load into a slot that is
    // not read again), so no load depends on a branch.
    auto step = [&](int t, auto sync) {
      const int rs = (t + 1) & 1;
      const u16* rdK = sK[rs];
      const u16* rdV = sV[rs];
      if (pend) {             // the reference moved at the previous step
#pragma unroll
        for (int d = 0; d < ND; ++d)
#pragma unroll
          for (int e = 0; e < 16; ++e) o[d][e] *= pend_alpha;
        pend = false;
      }
      uint32_t kbyte = (uint32_t)kbase(t + 2 < nf ? t + 2 : nf - 1) * (uint32_t)(D * 2);
      uint32_t vbyte = (uint32_t)kbase(t) * (uint32_t)(D * 2);
      if constexpr (SPARSE) {
        // Both entries are read before the window moves, so no read waits
        // for the chunk load below.  Entries advance by at most two per step
        // and K runs at most three entries ahead of V, so moving on once V
        // leaves chunk c0 keeps both inside the window; the chunk loaded
        // here is first read about 60 steps later.
        asm volatile("" : "+s"(kbyte), "+s"(vbyte));
        if ((entry(t) >> 6) > c0) {
          cid0 = cid1;
          cid1 = load_chunk(c0 + 2);
          ++c0;
        }
      }
      // LDS address of the slot being filled, re-derived every step: stops
      // the compiler from keeping one destination register per load across
      // the loop (which overflows the scalar registers).
      uint32_t fill = lds_addr(sKV[t & 1]);
      asm volatile("" : "+s"(fill));
      const uint32_t mbyte = ld.mixed_v ? vbyte : kbyte;
      auto loads = [&](int slot) {
        // Load n goes to slot n * SPAN / PW (at most one per slot): the
        // loads fill the first 5/16 of the step, so the last of them has
        // most of the step to land before the wait at its end.
        constexpr int PW = LD::PW, SPAN = (2 * NK + 4 * ND) * 5 / 16;
        static_assert(PW <= SPAN, "one load instruction per slot at most");
        const int n = (slot * PW + SPAN - 1) / SPAN;
        if (n >= PW || (n * SPAN) / PW != slot) return;
        ld.issue_n(n, fill, rKw, rVw, rMw, kbyte, vbyte, mbyte);
      };
      auto hook = [&](int slot) {
        loads(slot);
        if constexpr (BS)
          if (slot == (2 * NK + 4 * ND) / 2) flush_waiting();
      };
      f32x16 s_next[2];
      bf16x8 p_cur[2][2];
      float tsum = 0.f;
      pipelined_step<D, KS, VS, 2, BS, !SPARSE>(hook, rdK + klane, rdV + voff, qf, s_cur, p_prev, s_next, p_cur, o,
                                       sl2, ref.mc, rsum, &tsum);
      move_reference<2, BS>(ref, rsum, bad, s_cur, p_cur, pend, pend_alpha, sl2, c32, false, &tsum);
      if constexpr (BS) {
        if (pend) {                     // the reference moved at this tile
          bsum *= pend_alpha;
          rowf *= pend_alpha;
        }
        bsum += tsum;
        rowf += tsum;
        if (((t + 1) & (tpb - 1)) == 0) {
          bdone = bsum;
          cdone = t >> tsh;
          bsum = 0.f;
        }
      }
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        s_cur[g] = s_next[g];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) p_prev[g][s2] = p_cur[g][s2];
      }
      if (decltype(sync)::value) {
        wait_vmem();
        __syncthreads();
      }
    };
    int t = 0;
    for (; t + 1 < nf; t += 2) {
      step(t, std::true_type{});
      step(t + 1, std::true_type{});
    }
    if (t < nf) step(t, std::true_type{});
    flush_waiting();
    if (pend) {
#pragma unroll
      for (int d = 0; d < ND; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[d][e] *= pend_alpha;
    }
    pv_tile<ND, VS>(sV[(nf - 1) & (RING - 1)] + voff, p_prev, o);
    lsum = finish_sums(rsum, bad, p_prev, hw, c32);
    bad = bad || !acc_finite<ND>(o);
    redo = __any(bad);
    if (redo && lane == 0) s_redo = 1;
    __syncthreads();
  }
  const bool any_redo = s_redo != 0;
  if (redo) {
    ref = RowRef{};
    lsum = 0.f;
    bsum = 0.f;
    rowf = 0.f;
#pragma unroll
    for (int d = 0; d < ND; ++d) o[d] = f32x16{};
  }

  // Remaining tiles, one at a time with key masking (the waves that do not
  // compute a tile still issue their share of its loads and meet at the
  // barriers).
  auto masked_tile = [&](int kb, bool compute) {
    KDMA::issue(rK, sK[0], kb, wave, lane);
    VDMA::issue(rV, sV[0], kb, wave, lane);
    wait_vmem();
    __syncthreads();
    if (compute) {
      f32x16 s[2];
      qk_tile<D, KS>(sK[0], qf, c32, hw, s);
      mask_tile(s, L - kb, hw);
      bf16x8 pb[2][2];
      float alpha;
      if constexpr (BS) {
        float fs;
        alpha = softmax_tile_fsum(s, ref, lsum, sl2, pb, fs);
        bsum = bsum * alpha + fs;
        rowf = rowf * alpha + fs;
      } else {
        alpha = softmax_tile(s, ref, lsum, sl2, pb);
      }
#pragma unroll
      for (int d = 0; d < ND; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[d][e] *= alpha;
      pv_tile<ND, VS>(sV[0] + voff, pb, o);
    }
    __syncthreads();
  };
  if constexpr (SPARSE) {
    // Malformed rows: every entry; otherwise the tiles of the ragged block
    // the pipeline left out, and every tile for the waves that redo their
    // rows (in row order either way).
    auto entry_tiles = [&](int i) {
      const int c = a.col_idx[e0 + i];
      if (c < 0 || c >= a.nkb) return;
      for (int j = 0; j < sub; ++j) {
        const int kb = c * a.block + j * KT;
        const bool left = slow || (i == skip && j >= rag_sub);
        if (kb < L && (left || any_redo)) masked_tile(kb, left || redo);
      }
    };
    if (slow || any_redo) {
      for (int i = 0; i < ne; ++i) entry_tiles(i);
    } else if (skip >= 0) {
      entry_tiles(skip);
    }
    if (nf == 0 && spec >= 0) wait_vmem();    // no guessed load is left in flight
  } else {
    if (any_redo)
      for (int t = 0; t < nf; ++t) {
        masked_tile(t * KT, redo);
        if (redo && ((t + 1) & (tpb - 1)) == 0) flush_block(t >> tsh);
      }
    if (nf * KT < L) masked_tile(nf * KT, true);
    // The last key block: the ragged tile, or full tiles that stopped short
    // of a whole block.
    if (nf * KT < L || (nf & (tpb - 1)) != 0) flush_block(nf >> tsh);
  }

  // Normalise and store.
  float lt;
  {
    float lo, hi;
    half_pair(lsum, lo, hi);
    lt = lo + hi;
  }
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  // Every wave's tile loads have landed and its reads of the ring are done.
  static_assert(kStageElems<D, NW> <= RING * LD::ELEMS, "the output tiles fit the ring");
  __syncthreads();
  store_rows<D>(o, inv, &sKV[0][0] + wave * 32 * (D + 8), a.o + hoff, qt * (32 * NW) + wave * 32, L, lane);
  if (qrow < L && hw == 0 && a.lse != nullptr)
    a.lse[(size_t)bh * L + qrow] = lt > 0.f ? fmaf(ref.m, a.scale, logf(lt)) : -INFINITY;
  // The row's Q fragments, its sum and reference (LSE = m * scale + log lt)
  // and the K/V ring, which no wave reads any more after the next barrier.
  // With BS: the unrounded row sum and the reference in log2 units instead
  // (log2 e * LSE = mc + log2 of that sum, up to fp32 rounding).
  if constexpr (BS) {
    float lo, hi;
    half_pair(rowf, lo, hi);
    tail(bh, qt, qf, lo + hi, ref.mc, &sKV[0][0]);
  } else {
    tail(bh, qt, qf, lt, ref.m, &sKV[0][0]);
  }
}

template <int D, int NW, bool SPARSE>
__global__ __launch_bounds__(64 * NW, NW >= 8 ? 1 : 2) void attn_fwd_kernel(AttnParams a) {
  attn_fwd_body<D, NW, SPARSE>(a, NoTail{});
}

// ---------------------------------------------------------------------------
// Block-sparse attention with block 64, two query blocks per workgroup.
//
// Four waves cover query blocks 2P (waves 0-1) and 2P+1 (waves 2-3), 128
// rows, through the same pipeline as attn_fwd_kernel (one 64-key tile per
// block).  A byte map in LDS marks which row keeps each key block.  When both
// rows keep blocks the other does not, in similar numbers, the walk has two
// phases: the shared blocks as full steps for all 128 rows, then the solo
// blocks of both rows side by side as 32-key half steps (rows 0-31 of a slot
// hold a half tile of one row's block, rows 32-63 one of the other's, and
// each half reads its own rows), so neither half computes on a tile it does
// not keep.  Otherwise the pair walks the sorted union in ascending order:
// for a tile that only one row keeps, the other half takes its probabilities
// against a reference of +inf, so they are exact zeros (exp2(-inf)) and each
// half accumulates exactly its own tiles, in ascending order, as a one-block
// workgroup would (this keeps all-blocks-kept bitwise equal to the dense
// kernel); that costs one scalar select per step (overwriting the scores
// with -inf made every step wait for its score MFMAs, ~7%).  A non-finite
// score in such a tile (an inf or NaN in a key the half does not keep)
// would still reach the half's sums; it leaves them, or the output
// accumulator, non-finite, which sends the wave to the exact path, where the
// tile's scores are masked to -inf before the softmax.  Rows must be
// strictly ascending lists of blocks in [0, NB); otherwise (or for the
// ragged last block) tiles are done one at a time with key masking.
// ---------------------------------------------------------------------------
template <int D, int NW>
__global__ __launch_bounds__(64 * NW, NW >= 8 ? 1 : 2) void attn_sparse_pair_kernel(AttnParams a) {
  constexpr int NT = 64 * NW;
  constexpr int WPB = NW / 2;        // waves per query block
  constexpr int BLK = 32 * WPB;      // block size: 64 (four waves) or 128 (eight waves)
  constexpr int SUB = BLK / KT;      // 64-key tiles per block
  using KDMA = TileDMA<D, NW, 1>;
  using VDMA = TileDMA<D, NW, 2>;
  constexpr int KS = KDMA::S, VS = VDMA::S;
  constexpr int ND = D / 32;
  constexpr int NK = D / 16;
  using LD = KVLoader<D, NW>;
  __shared__ __attribute__((aligned(1024))) u16 sKV[2][LD::ELEMS];   // slots [K | V]
  __shared__ uint8_t sMap[kMaxBlocks];                                 // the rows' block map
  const SlotPart<LD::ELEMS, 0> sK{sKV};
  const SlotPart<LD::ELEMS, LD::VOFF> sV{sKV};

  int bh, pq;
  {
    int item = (int)blockIdx.x;
    if (item >= a.n_static) {                // as in attn_fwd_kernel
      __shared__ int s_tail;
      if (threadIdx.x == 0) s_tail = claim_item<true>(a.claim, a.n_static, a.n_items);
      __syncthreads();
      item = s_tail;
      if (item < 0) return;
    }
    text_first_map(item, a.n_items, a.nqt, a.tq0, a.tq1 - a.tq0, bh, pq);
  }
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int mybit = 1 << (wave / WPB);                         // 1: row 2P, 2: row 2P+1
  const int hw = lane >> 5, c32 = lane & 31;
  const int gi = lane & 15, grp = lane >> 4;
  const int L = a.seqlen, nkb = a.nkb;
  const size_t hoff = (size_t)bh * L * D;
  const uint32_t hbytes = (uint32_t)L * D * 2u;
  const __amdgpu_buffer_rsrc_t rK = make_rsrc(a.k + hoff, hbytes);
  const __amdgpu_buffer_rsrc_t rV = make_rsrc(a.v + hoff, hbytes);
  const u32x4 rKw = rsrc_words(a.k + hoff, hbytes), rVw = rsrc_words(a.v + hoff, hbytes);
  const int qrow = pq * (2 * BLK) + wave * 32 + c32;
  const int voff = ((4 * hw + (gi >> 2)) * VS) * 8 + 16 * (grp & 1) + 4 * (gi & 3);
  const int klane = (c32 * KS + hw) * 8;

#pragma unroll
  for (int b = 0; b < 2; ++b) zero_lds<VDMA::SLOTS>(sV[b], tid, NT);   // finite V
  bf16x8 qf[NK];
  load_q<D>(a.q + hoff, qrow, L, hw, qf);
  // As in attn_fwd_kernel: under the text sink the union of the two rows
  // begins with the text blocks, so its first two tiles are loaded on a guess
  // before the indices are read (checked before the first tile is used).
  const int g0 = a.kb_guess >= 0 ? a.kb_guess * BLK : -1;
  const int g1 = g0 < 0 ? -1 : (SUB > 1 ? g0 + KT : (a.n_guess >= 2 ? g0 + BLK : -1));
  if (g0 >= 0) KDMA::issue(rK, sK[0], g0, wave, lane);
  if (g1 >= 0) KDMA::issue(rK, sK[1], g1, wave, lane);

  // The two rows.  Each row's indices are read 64 at a time into one
  // register per lane through a resource bounded to the row (lanes past its
  // end read 0), as in attn_fwd_kernel.
  int len[2], beg[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int p = 2 * pq + r;
    int64_t s0 = 0, e0 = 0;
    if (p < nkb) {
      const int64_t row = (int64_t)bh * nkb + p;
      s0 = a.row_ptr[row];
      e0 = a.row_ptr[row + 1];
      s0 = s0 < 0 ? 0 : (s0 > a.col_count ? a.col_count : s0);
      e0 = e0 < s0 ? s0 : (e0 > a.col_count ? a.col_count : e0);
    }
    beg[r] = (int)s0;
    len[r] = (int)(e0 - s0);
  }
  const __amdgpu_buffer_rsrc_t rC0 = make_rsrc(a.col_idx + beg[0], (uint32_t)len[0] * 4u);
  const __amdgpu_buffer_rsrc_t rC1 = make_rsrc(a.col_idx + beg[1], (uint32_t)len[1] * 4u);
  auto load_chunk = [&](int r, int c) -> int {
    return __builtin_amdgcn_raw_buffer_load_b32(r == 0 ? rC0 : rC1, (uint32_t)(c * 64 + lane) * 4u, 0, 0);
  };
  // Two-chunk windows of each row, loaded first; the prologue's scans read
  // chunks 0 and 1 from them.
  int w0[2], w1[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    w0[r] = load_chunk(r, 0);
    w1[r] = load_chunk(r, 1);
  }
  auto chunk = [&](int r, int c) -> int { return c == 0 ? w0[r] : (c == 1 ? w1[r] : load_chunk(r, c)); };
  // Validation: every entry in [0, NB) and each row strictly ascending;
  // whether a row keeps the ragged last block (always its last entry).
  const bool ragged_L = L % BLK != 0;
  bool slow = false;
  int rag = 0;                        // bit r: row r keeps the ragged block
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    int last = -1;
    for (int c = 0; c * 64 < len[r]; ++c) {
      const int n = c * 64 + lane;
      const int v = chunk(r, c);
      int prev = __shfl_up(v, 1, 64);
      if (lane == 0) prev = last;
      const bool valid = n < len[r];
      if (__any(valid && (v < 0 || v >= nkb || v <= prev))) slow = true;
      if (__any(valid && ragged_L && v == nkb - 1)) rag |= 1 << r;
      last = __builtin_amdgcn_readlane(v, 63);
    }
  }
  // Byte map of the two rows' key blocks (bit 0: block 2P keeps it, bit 1:
  // block 2P+1 keeps it), without the ragged block (done masked at the end).
  // Shared blocks run as full steps for all 128 rows (phase 1); the blocks
  // only one row keeps run afterwards as dual half steps (phase 2): each
  // step holds 32 keys of one solo block of each row, so neither half
  // computes for a tile it does not keep.
  static_assert(SUB == 1, "one 64-key tile per block");
  int n_shared = 0;
  if (!slow) {
    for (int i = tid; i < nkb; i += NT) sMap[i] = 0;
    __syncthreads();
    for (int c = 0; c * 64 < len[0]; ++c) {
      const int v = chunk(0, c);
      if (c * 64 + lane < len[0] && !(ragged_L && v == nkb - 1)) sMap[v] = 1;
    }
    __syncthreads();
    // Every wave writes the same value (bit 0 is final after the barrier
    // and kept), so the waves' writes agree whatever their order, and every
    // wave counts the same shared blocks from bit 0.
    for (int c = 0; c * 64 < len[1]; ++c) {
      const int v = chunk(1, c);
      const bool in = c * 64 + lane < len[1] && !(ragged_L && v == nkb - 1);
      const int a_keeps = in ? (sMap[v] & 1) : 0;
      if (in) sMap[v] = (uint8_t)(a_keeps | 2);
      n_shared += __builtin_popcountll(__ballot(a_keeps != 0));
    }
  }
  // Dual half steps pay off when both rows have solo blocks in similar
  // numbers (a half step costs a little over half a full step).  Otherwise
  // (one row has none, as for the single block of the last pair when NB is
  // odd, or a text row beside a video row) phase 1 walks the whole union in
  // ascending order instead, the half that does not keep a tile taking it
  // hidden, and there is no phase 2.
  const int na = len[0] - (rag & 1), nb = len[1] - ((rag >> 1) & 1);
  const int nAs = na - n_shared, nBs = nb - n_shared;
  const int s_min = nAs < nBs ? nAs : nBs, s_max = nAs < nBs ? nBs : nAs;
  const bool dual = !slow && s_min > 0 && s_min * 6 > s_max;
  const int nf1 = slow ? 0 : (dual ? n_shared : na + nb - n_shared);   // phase 1: full steps
  const int cls1 = dual ? 3 : 0;                           // its blocks: shared, or the union
  const int nA2 = dual ? 2 * nAs : 0;                      // phase 2: half tiles of each row
  const int nB2 = dual ? 2 * nBs : 0;
  const int nf2 = nA2 > nB2 ? nA2 : nB2;
  const int half = wave / WPB;                             // 0: block 2P, 1: block 2P+1
  const int n_mine = half == 0 ? nA2 : nB2;

  // Blocks of one class of the map in ascending order (cls 3: both rows keep
  // it, 1 or 2: only that row, 0: either), 64 map entries at a time (ballots
  // over the window, then the set bits); -1 when exhausted.  keep receives
  // the block's map entry.
  struct MapStream {
    int w;
    uint64_t m, ma, mb;
  };
  const int nwin = (nkb + 63) / 64;
  auto next_of = [&](MapStream& st, int cls, int& keep) -> int {
    while (st.m == 0ull) {
      if (++st.w >= nwin) return -1;
      const int blk = st.w * 64 + lane;
      const int v = blk < nkb ? sMap[blk] : 0;
      st.ma = __ballot((v & 1) != 0);
      st.mb = __ballot((v & 2) != 0);
      st.m = cls == 0 ? (st.ma | st.mb)
                      : (cls == 3 ? (st.ma & st.mb) : (cls == 1 ? (st.ma & ~st.mb) : (st.mb & ~st.ma)));
    }
    const int j = __builtin_ctzll(st.m);
    st.m &= st.m - 1;
    keep = (int)((st.ma >> j) & 1ull) | ((int)((st.mb >> j) & 1ull) << 1);
    return st.w * 64 + j;
  };

  const float sl2 = a.scale_log2;
  RowRef ref;
  float lsum = 0.f;
  f32x16 o[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d) o[d] = f32x16{};
  auto hide = [&](f32x16 (&s)[2]) {   // this half does not keep the tile
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[g][e] = -INFINITY;
  };
  __shared__ int s_redo;              // as in attn_fwd_kernel
  if (tid == 0) s_redo = 0;
  bool redo = false;
  __syncthreads();                    // the map is complete

  bf16x8 p_prev[2][2];
  bool pend = false;
  float pend_alpha = 1.f;
  RowSums rsum;
  rsum.init(lane);
  bool bad = false;
  LD ld;
  ld.init(wave, lane);
  const u32x4 rMw = ld.mixed_v ? rVw : rKw;     // resource of this wave's mixed entry
  auto rescale_pending = [&]() {
    if (pend) {             // the reference moved at the previous step
#pragma unroll
      for (int d = 0; d < ND; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[d][e] *= pend_alpha;
      pend = false;
    }
  };

  if (nf1 > 0) {
    // Phase 1: blocks u0 = t, t + 1, t + 2 at step t (block, map entry), as
    // in attn_fwd_kernel.
    MapStream ss{-1, 0ull, 0ull, 0ull};
    int ub[3], uk[3] = {0, 0, 0};
#pragma unroll
    for (int j = 0; j < 3; ++j) ub[j] = next_of(ss, cls1, uk[j]);
    int u0 = 0;
    auto pick = [&](int slot) { return slot == 0 ? ub[0] : (slot == 1 ? ub[1] : ub[2]); };
    auto tile_row = [&](int j) { return pick(j - u0) * BLK; };    // j within the queue's reach
    const int r0 = tile_row(0), r1 = nf1 > 1 ? tile_row(1) : -1;
    if (!(g0 >= 0 && r0 == g0 && (nf1 < 2 || r1 == g1))) {
      if (g0 >= 0) wait_vmem();          // this wave's guessed loads land first
      KDMA::issue(rK, sK[0], r0, wave, lane);
      if (nf1 > 1) KDMA::issue(rK, sK[1], r1, wave, lane);
    }
    wait_vmem();
    __syncthreads();
    f32x16 s_cur[2];
    qk_tile<D, KS>(sK[0], qf, c32, hw, s_cur);
    bool hid = !(uk[0] & mybit);
    __syncthreads();                  // sK[0] is refilled by step 0
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) p_prev[g][s2] = bf16x8{};

    auto step = [&](int t, auto rs_c) {
      constexpr int RS = decltype(rs_c)::value;
      rescale_pending();
      uint32_t kbyte = (uint32_t)tile_row(t + 2 < nf1 ? t + 2 : nf1 - 1) * (uint32_t)(D * 2);
      uint32_t vbyte = (uint32_t)tile_row(t) * (uint32_t)(D * 2);
      asm volatile("" : "+s"(kbyte), "+s"(vbyte));
      uint32_t fill = lds_addr(sKV[1 - RS]);
      asm volatile("" : "+s"(fill));
      const uint32_t mbyte = ld.mixed_v ? vbyte : kbyte;
      auto loads = [&](int slot) {
        constexpr int PW = LD::PW, SPAN = (2 * NK + 4 * ND) * 5 / 16;   // as in attn_fwd_kernel
        static_assert(PW <= SPAN, "one load instruction per slot at most");
        const int n = (slot * PW + SPAN - 1) / SPAN;
        if (n >= PW || (n * SPAN) / PW != slot) return;
        ld.issue_n(n, fill, rKw, rVw, rMw, kbyte, vbyte, mbyte);
      };
      f32x16 s_next[2];
      bf16x8 p_cur[2][2];
      pipelined_step<D, KS, VS>(loads, sK[RS] + klane, sV[RS] + voff, qf, s_cur, p_prev, s_next, p_cur, o,
                                sl2, hid ? INFINITY : ref.mc, rsum);
      move_reference(ref, rsum, bad, s_cur, p_cur, pend, pend_alpha, sl2, c32, hid);
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        s_cur[g] = s_next[g];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) p_prev[g][s2] = p_cur[g][s2];
      }
      hid = !(uk[1] & mybit);          // tile t+1
      ub[0] = ub[1];
      uk[0] = uk[1];
      ub[1] = ub[2];
      uk[1] = uk[2];
      if (u0 + 3 < nf1) ub[2] = next_of(ss, cls1, uk[2]);
      ++u0;
      wait_vmem();
      __syncthreads();
    };
    int t = 0;
    for (; t + 1 < nf1; t += 2) {
      step(t, std::integral_constant<int, 1>{});
      step(t + 1, std::integral_constant<int, 0>{});
    }
    if (t < nf1) step(t, std::integral_constant<int, 1>{});
    rescale_pending();
    pv_tile<ND, VS>(sV[(nf1 - 1) & 1] + voff, p_prev, o);
#pragma unroll
    for (int j = 0; j < 4; ++j) rsum.add(p_prev[j >> 1][j & 1]);
    bad = bad || !(rsum.acc[0] <= kRowSumBad);
  }

  if (nf2 > 0) {
    // Phase 2: dual half steps.  Half tile t of a row is keys [32 (t % 2),
    // 32 (t % 2) + 32) of its (t / 2)-th solo block; rows [0, 32) of a slot
    // hold block 2P's half tile, rows [32, 64) block 2P+1's, and each half of
    // the workgroup reads its own rows.  A row with fewer half tiles than the
    // other takes its surplus steps hidden (key 0 loaded in their place).
    if (nf1 == 0 && g0 >= 0) wait_vmem();   // the guessed loads land before these
    MapStream sa{-1, 0ull, 0ull, 0ull}, sb{-1, 0ull, 0ull, 0ull};
    int qa[2], qb[2], kp;                    // solo blocks of half tiles t and t + 2
    qa[0] = next_of(sa, 1, kp);
    qa[1] = next_of(sa, 1, kp);
    qb[0] = next_of(sb, 2, kp);
    qb[1] = next_of(sb, 2, kp);
    auto key = [](int t, int n, int blk) { return t < n ? blk * BLK + 32 * (t & 1) : 0; };
    TileDMA<D, NW, 1>::issue_dual(rK, sK[0], key(0, nA2, qa[0]), key(0, nB2, qb[0]), wave, lane);
    TileDMA<D, NW, 1>::issue_dual(rK, sK[1], key(1, nA2, qa[0]), key(1, nB2, qb[0]), wave, lane);
    wait_vmem();
    __syncthreads();
    const int klane_h = klane + half * 32 * KS * 8;
    const int voff_h = voff + half * 32 * VS * 8;
    const uint32_t hmask = LD::half_mask(wave, lane);
    f32x16 s_cur[2];
    qk_tile<D, KS, 1>(sK[0] + klane_h - klane, qf, c32, hw, s_cur);
    bool hid = 0 >= n_mine;
    __syncthreads();                  // sK[0] is refilled by step 0
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) p_prev[0][s2] = bf16x8{};

    auto step2 = [&](int t, auto rs_c) {
      constexpr int RS = decltype(rs_c)::value;
      rescale_pending();
      constexpr uint32_t HALF_BYTES = 32u * D * 2u;
      uint32_t ka = (uint32_t)key(t + 2, nA2, qa[1]) * (uint32_t)(D * 2);
      uint32_t kb = (uint32_t)key(t + 2, nB2, qb[1]) * (uint32_t)(D * 2) - HALF_BYTES;
      uint32_t va = (uint32_t)key(t, nA2, qa[0]) * (uint32_t)(D * 2);
      uint32_t vb = (uint32_t)key(t, nB2, qb[0]) * (uint32_t)(D * 2) - HALF_BYTES;
      asm volatile("" : "+s"(ka), "+s"(kb), "+s"(va), "+s"(vb));
      uint32_t fill = lds_addr(sKV[1 - RS]);
      asm volatile("" : "+s"(fill));
      auto loads = [&](int slot) {      // loads in the first PW slots of the step
        constexpr int PW = LD::PW;
        if (slot >= PW) return;
        ld.issue_dual_n(slot, fill, rKw, rVw, rMw, ka, kb, va, vb, hmask);
      };
      f32x16 s_next[2];
      bf16x8 p_cur[2][2];
      pipelined_step<D, KS, VS, 1>(loads, sK[RS] + klane_h, sV[RS] + voff_h, qf, s_cur, p_prev, s_next,
                                   p_cur, o, sl2, hid ? INFINITY : ref.mc, rsum);
      move_reference<1>(ref, rsum, bad, s_cur, p_cur, pend, pend_alpha, sl2, c32, hid);
      s_cur[0] = s_next[0];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) p_prev[0][s2] = p_cur[0][s2];
      hid = t + 1 >= n_mine;
      if (t & 1) {                        // half tile t was the second of its block
        qa[0] = qa[1];
        qa[1] = next_of(sa, 1, kp);
        qb[0] = qb[1];
        qb[1] = next_of(sb, 2, kp);
      }
      wait_vmem();
      __syncthreads();
    };
    int t = 0;
    for (; t + 1 < nf2; t += 2) {
      step2(t, std::integral_constant<int, 1>{});
      step2(t + 1, std::integral_constant<int, 0>{});
    }
    if (t < nf2) step2(t, std::integral_constant<int, 1>{});
    rescale_pending();
    pv_tile<ND, VS, 1>(sV[(nf2 - 1) & 1] + voff_h, p_prev, o);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) rsum.add(p_prev[0][s2]);
    bad = bad || !(rsum.acc[0] <= kRowSumBad);
  }

  if (nf1 + nf2 > 0) {
    const float v = RowSums::for_row(rsum.acc[0], c32);
    lsum = hw == 0 ? v : 0.f;
    bad = bad || !acc_finite<ND>(o);
    redo = __any(bad);
    if (redo && lane == 0) s_redo = 1;
    __syncthreads();
  }
  const bool any_redo = s_redo != 0;
  if (redo) {
    ref = RowRef{};
    lsum = 0.f;
#pragma unroll
    for (int d = 0; d < ND; ++d) o[d] = f32x16{};
  }

  // One tile with key masking, kept by the rows in keep (computed by the
  // waves in compute; the others only load and meet at the barriers).
  auto masked_tile = [&](int kb, int keep, bool compute) {
    KDMA::issue(rK, sK[0], kb, wave, lane);
    VDMA::issue(rV, sV[0], kb, wave, lane);
    wait_vmem();
    __syncthreads();
    if (compute) {
      f32x16 s[2];
      qk_tile<D, KS>(sK[0], qf, c32, hw, s);
      mask_tile(s, L - kb, hw);
      if (!(keep & mybit)) hide(s);
      bf16x8 pb[2][2];
      const float alpha = softmax_tile(s, ref, lsum, sl2, pb);
#pragma unroll
      for (int d = 0; d < ND; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[d][e] *= alpha;
      pv_tile<ND, VS>(sV[0] + voff, pb, o);
    }
    __syncthreads();
  };
  if (slow || any_redo) {
    // Malformed rows, or waves that redo their rows: each row's valid
    // entries in its own order.
#pragma unroll
    for (int r = 0; r < 2; ++r)
      for (int i = 0; i < len[r]; ++i) {
        const int c = a.col_idx[beg[r] + i];
        if (c >= 0 && c < nkb)
          for (int j = 0; j < SUB; ++j)
            if (c * BLK + j * KT < L) masked_tile(c * BLK + j * KT, 1 << r, slow || redo);
      }
  }
  if (!slow && rag) {
    for (int j = 0; j < SUB; ++j)
      if ((nkb - 1) * BLK + j * KT < L) masked_tile((nkb - 1) * BLK + j * KT, rag, !redo);
  }
  if (nf1 + nf2 == 0 && g0 >= 0) wait_vmem();   // no guessed load is left in flight

  float lt;
  {
    float lo, hi;
    half_pair(lsum, lo, hi);
    lt = lo + hi;
  }
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  // As in attn_fwd_body: the output tiles go out through the free ring.
  static_assert(kStageElems<D, NW> <= 2 * LD::ELEMS, "the output tiles fit the ring");
  __syncthreads();
  store_rows<D>(o, inv, &sKV[0][0] + wave * 32 * (D + 8), a.o + hoff, pq * (2 * BLK) + wave * 32, L, lane);
  if (qrow < L && hw == 0 && a.lse != nullptr)
    a.lse[(size_t)bh * L + qrow] = lt > 0.f ? fmaf(ref.m, a.scale, logf(lt)) : -INFINITY;
}

// ---------------------------------------------------------------------------
// Block attention mass: W[p][c] = sum_{i in p, j in c} exp(scale*q_i.k_j - LSE_i)
//
// One workgroup of eight waves (32 rows each) covers 256 query rows: QB
// adjacent query blocks (two of 128 or four of 64), so every K tile brought
// into LDS serves 256 rows, and two workgroups share a CU (four waves per
// SIMD: the pass needs under 128 registers).  Against workgroups of 128 rows
// this halves the tile traffic per FLOP; the pass is bound by its QK MFMAs
// at the clock the chip's power allows (the exponentials hide under the
// other waves' MFMAs), so the saving shows as clock (110K: 67.1 -> 65.1 ms
// at block 128, 70.3 -> 68.9 ms at block 64, masses bitwise unchanged).
// Full key tiles run through a software pipeline: step t forms the scores of tile t+1 (QK MFMAs) while the
// VALU exponentiates and sums tile t; K is double-buffered and the loads of
// tile t+2 are spread over the step.  Per-wave sums of a finished key block
// are combined in a fixed order into an LDS ring per query block, which is
// written out 64 blocks at a time (coalesced).
// ---------------------------------------------------------------------------
constexpr int kMassRing = 128;        // blocks of W per row held in LDS before they are written out

// The mass pass of query-block group pg of head bh (QB query blocks, 256
// rows).  qsrc(qf, nlse2, hoff, qrow, qvalid, hw) supplies this lane's Q
// fragments and -LSE * log2(e) of its row (-inf for a row past L, whose
// exp2 terms are then 0); sK0 / sK1 are the two K tile buffers, sRed the
// per-wave sums of the last two blocks and sW the ring of W blocks not yet
// written out.
template <int D, int QB, int NW, typename QSrc>
__device__ __forceinline__ void block_mass_body(const MassParams& a, int bh, int pg, QSrc&& qsrc,
                                                u16* sK0, u16* sK1, float (*sRed)[NW],
                                                float (*sW)[kMassRing]) {
  constexpr int NT = 64 * NW;
  constexpr int WPB = NW / QB;       // waves per query block
  constexpr int SUB = 32 * WPB / KT; // KT-key tiles per key block
  using KDMA = TileDMA<D, NW, 1>;
  constexpr int KS = KDMA::S;
  constexpr int NK = D / 16;
  constexpr int RING = kMassRing, CHUNK = 64;

  const int p0 = pg * QB;           // first query block of the group
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int hw = lane >> 5, c32 = lane & 31;
  const int L = a.seqlen;
  const size_t hoff = (size_t)bh * L * D;
  const __amdgpu_buffer_rsrc_t rK = make_rsrc(a.k + hoff, (uint32_t)L * D * 2u);
  const u32x4 rKw = rsrc_words(a.k + hoff, (uint32_t)L * D * 2u);
  const int qrow = pg * (32 * NW) + wave * 32 + c32;
  const bool qvalid = qrow < L;

  bf16x8 qf[NK];
  float nlse2;
  qsrc(qf, nlse2, hoff, qrow, qvalid, hw);
  const float sl2 = a.scale_log2;
  const int sub = SUB;
  const int nfull = L / KT;   // full key tiles
  float* wrow = a.w + ((size_t)bh * a.nkb + p0) * a.nkb;    // row p0 + qb at wrow + qb * nkb
  const int nrows = a.nkb - p0 < QB ? a.nkb - p0 : QB;      // rows of W this group owns

  float acc = 0.f;
  auto reduce_block = [&](float v, int blk) {
    const float w = wave_sum(v);
    if (lane == 0) sRed[blk & 1][wave] = w;
  };
  auto finish_block = [&](int blk) {
    reduce_block(acc, blk);
    acc = 0.f;
  };
  // Pipelined tiles: the sum of a key block that ended at step t waits in
  // adone and is reduced over the wave in the middle of step t + 1, under
  // its MFMAs, so the end of step t does not wait for that chain; it is
  // published after step t + 1's barrier.  bdone is its block, -1 when none
  // waits; npub counts the blocks published so far.
  float adone = 0.f;
  int bdone = -1;
  int npub = 0;
  // After a barrier: waves combined in a fixed order (deterministic).
  auto publish = [&](int blk) {
    if (tid == 0) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float v = 0.f;
#pragma unroll
        for (int w = qb * WPB; w < (qb + 1) * WPB; ++w) v += sRed[blk & 1][w];
        sW[qb][blk % RING] = v;
      }
    }
  };
  // After a barrier that follows the publication of block blk: once a chunk
  // of CHUNK blocks is complete, write it out (it is not touched again until
  // the ring wraps, CHUNK blocks and at least one barrier later).
  int flushed = 0;                  // blocks [0, flushed) written out
  auto flush = [&](int done) {      // blocks [0, done) published
    while (done - flushed >= CHUNK) {
      if (tid < CHUNK * QB) {
        const int qb = tid / CHUNK, i = flushed + tid % CHUNK;
        if (qb < nrows) wrow[(size_t)qb * a.nkb + i] = sW[qb][i % RING];
      }
      flushed += CHUNK;
    }
  };
  __syncthreads();

  if (nfull > 0) {
    KDMA::issue(rK, sK0, 0, wave, lane);
    if (nfull > 1) KDMA::issue(rK, sK1, KT, wave, lane);
    wait_vmem();
    __syncthreads();
    f32x16 s_cur[2];
    qk_tile<D, KS>(sK0, qf, c32, hw, s_cur);
    __syncthreads();            // sK0 is refilled by step 0

    KLoader<D, NW> ld;
    ld.init(wave, lane);
    const int klane = (c32 * KS + hw) * 8;
    // Step t (t + 1 < nfull) sums tile t, forms the scores of tile t+1 from
    // buffer (t+1)&1 and loads tile t+2 into buffer t&1.
    // Past the last tile the load is clamped to the last one (an in-range
    // load into a buffer that is not read again), so no load is branched.
    auto step = [&](int t, const u16* rdK, u16* ldK) {
      const uint32_t kbyte = (uint32_t)(t + 2 < nfull ? t + 2 : nfull - 1) * (uint32_t)(KT * D * 2);
      uint32_t fill = lds_addr(ldK);
      asm volatile("" : "+s"(fill));
      auto loads = [&](int slot) {
        // Load n goes to slot n * NM / NTOT: spread over the whole step here
        // (front-loaded as in attn_fwd_kernel this pass, with twice the
        // VALU work per MFMA, ran 3-5% slower).
        constexpr int NTOT = KLoader<D, NW>::PW, NM = 2 * NK;
        static_assert(NTOT <= NM, "one load instruction per slot at most");
        const int n = (slot * NTOT + NM - 1) / NM;
        if (n >= NTOT || (n * NM) / NTOT != slot) return;
        ld.issue_n(n, fill, rKw, kbyte);
      };
      auto hook = [&](int slot) {
        loads(slot);
        if (slot == NK && bdone >= 0) reduce_block(adone, bdone);
      };
      f32x16 s_next[2];
      mass_step<D, KS>(hook, rdK + klane, qf, s_cur, s_next, acc, sl2, nlse2);
      s_cur[0] = s_next[0];
      s_cur[1] = s_next[1];
      const int reduced = bdone;
      bdone = -1;
      if ((t + 1) % sub == 0) {
        adone = acc;
        acc = 0.f;
        bdone = t / sub;
      }
      wait_vmem();
      __syncthreads();
      flush(npub);                  // blocks published before this barrier
      if (reduced >= 0) {
        publish(reduced);
        npub = reduced + 1;
      }
    };
    int t = 0;
    for (; t + 2 < nfull; t += 2) {
      step(t, sK1, sK0);
      step(t + 1, sK0, sK1);
    }
    if (t + 1 < nfull) {
      step(t, sK1, sK0);
      ++t;
    }
    if (bdone >= 0) {
      reduce_block(adone, bdone);
      __syncthreads();
      publish(bdone);
      npub = bdone + 1;
      bdone = -1;
    }
    // Last full tile: its scores are in s_cur.
#pragma unroll
    for (int e = 0; e < 32; ++e) acc += fast_exp2(fmaf(s_cur[e >> 4][e & 15], sl2, nlse2));
    if ((t + 1) % sub == 0) {
      finish_block(t / sub);
      __syncthreads();
      publish(t / sub);
    }
  }
  // Ragged last tile (L not a multiple of KT), with key masking.
  if (nfull * KT < L) {
    __syncthreads();
    KDMA::issue(rK, sK0, nfull * KT, wave, lane);
    wait_vmem();
    __syncthreads();
    f32x16 s[2];
    qk_tile<D, KS>(sK0, qf, c32, hw, s);
    mask_tile(s, L - nfull * KT, hw);
#pragma unroll
    for (int e = 0; e < 32; ++e) acc += fast_exp2(fmaf(s[e >> 4][e & 15], sl2, nlse2));
  }
  // The last block, when its tiles did not end on a block boundary.
  if (nfull % sub != 0 || nfull * KT < L) {
    finish_block(a.nkb - 1);
    __syncthreads();
    publish(a.nkb - 1);
  }
  __syncthreads();
  for (int qb = 0; qb < nrows; ++qb)
    for (int i = flushed + tid; i < a.nkb; i += NT) wrow[(size_t)qb * a.nkb + i] = sW[qb][i % RING];
}

template <int D, int QB, int NW>
__global__ __launch_bounds__(64 * NW, 2) void block_mass_kernel(MassParams a) {
  using KDMA = TileDMA<D, NW, 1>;
  __shared__ __attribute__((aligned(1024))) u16 sK0[KDMA::ELEMS];
  __shared__ __attribute__((aligned(1024))) u16 sK1[KDMA::ELEMS];
  __shared__ float sRed[2][NW];           // per-wave sums of the last two blocks
  __shared__ float sW[QB][kMassRing];     // blocks of the QB rows of W not yet written out

  const int ngrp = (a.nkb + QB - 1) / QB;    // query-block groups per head
  // One contiguous range of (head, query-block group) items per XCD, through
  // the per-XCD work queues when a workspace is given (see claim_item).
  int bh, pg;
  {
    int item = (int)blockIdx.x;
    if (a.claim != nullptr) {
      __shared__ int s_item;
      if (threadIdx.x == 0) s_item = claim_item(a.claim, 0, a.n_items);
      __syncthreads();
      item = s_item;
      if (item < 0) return;
    }
    const int lid = xcd_remap(item, a.n_items);
    bh = lid / ngrp;
    pg = lid % ngrp;
  }
  auto qsrc = [&](bf16x8 (&qf)[D / 16], float& nlse2, size_t hoff, int qrow, bool qvalid, int hw) {
    load_q<D>(a.q + hoff, qrow, a.seqlen, hw, qf);
    // A padding row (past L) gets -inf: exp2 of it is 0 and it adds nothing.
    nlse2 = qvalid ? -a.lse[(size_t)bh * a.seqlen + qrow] * kLog2e : -INFINITY;
  };
  block_mass_body<D, QB, NW>(a, bh, pg, qsrc, sK0, sK1, sRed, sW);
}

// ---------------------------------------------------------------------------
// Fused online search (Algorithm 1) in one launch.  Each workgroup of eight
// waves takes 256 query rows of one head: the first pass is the dense
// attention of those rows (output and LSE, as attn_fwd_kernel<D, 8, false>),
// the second the block masses of the same rows (QB query blocks of
// 256 / QB rows, as block_mass_kernel<D, QB, 8>) against that LSE.  The
// second pass takes each row's Q fragments and LSE from the registers of the
// first instead of memory (the same lanes hold the same rows in both), and
// its LDS buffers are carved out of the attention ring, which is free once
// every wave has passed the barrier after its last read.  Both passes
// compute exactly what the two separate kernels compute.
// ---------------------------------------------------------------------------
template <int D, int QB>
__global__ __launch_bounds__(512, 1) void fused_search_kernel(AttnParams a, MassParams m) {
  constexpr int NW = 8;
  using LD = KVLoader<D, NW>;
  static_assert(TileDMA<D, NW, 1>::ELEMS <= LD::VOFF, "a mass K tile fits the K part of a ring slot");
  static_assert((2 * NW + QB * kMassRing) * 4 <= TileDMA<D, NW, 2>::ELEMS * 2,
                "the mass sums fit the V part of ring slot 0");
  attn_fwd_body<D, NW, false>(a, [&](int bh, int qt, const bf16x8 (&qf)[D / 16], float lt, float mref,
                                     u16* ring) {
    const float lse = lt > 0.f ? fmaf(mref, a.scale, logf(lt)) : -INFINITY;   // as stored
    __syncthreads();
    float* sums = reinterpret_cast<float*>(ring + LD::VOFF);
    auto qsrc = [&](bf16x8 (&q2)[D / 16], float& nlse2, size_t, int, bool qvalid, int) {
#pragma unroll
      for (int i = 0; i < D / 16; ++i) q2[i] = qf[i];
      nlse2 = qvalid ? -lse * kLog2e : -INFINITY;
    };
    block_mass_body<D, QB, NW>(m, bh, qt, qsrc, ring, ring + LD::ELEMS,
                               reinterpret_cast<float (*)[NW]>(sums),
                               reinterpret_cast<float (*)[kMassRing]>(sums + 2 * NW));
  });
}

// ---------------------------------------------------------------------------
// Single-pass online search (Algorithm 1 with one pass over Q K^T).  The mass
// of block (p, c) is the sum over rows i of p and keys j of c of
// exp(s_ij - LSE_i).  With the row's reference m_i (raw score units) that is
// the sum over i of exp2(ylog_ic - LSE_i log2 e), where ylog_ic = log2(sum_j
// exp2((s_ij - m_i) scale log2 e)) + m_i scale log2 e.  The attention pass
// takes every exp2((s_ij - m_i) scale log2 e) for its softmax anyway, so it
// adds their fp32 values per key block and writes ylog (attn_fwd_body with
// BS), and at the end of each row log2 e * LSE_i.  That LSE is the one of
// the unrounded fp32 row sum (the stored LSE normalises the bf16-rounded
// weights of the output), so each row's masses add up to one to fp32
// rounding.  A second kernel then streams ylog once and sums the rows'
// shares per block.  No second Q K^T is taken (the two-pass search
// recomputes it in full).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(512, 1) void single_pass_search_kernel(AttnParams a) {
  constexpr int NW = 8;
  attn_fwd_body<D, NW, false, true>(a, [&](int bh, int qt, const bf16x8 (&)[D / 16], float rowf, float mc,
                                           u16*) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int qrow = qt * (32 * NW) + wave * 32 + (lane & 31);
    // A row without weight adds nothing to any block.
    if (lane < 32 && qrow < a.seqlen)
      a.ylse2[(size_t)bh * a.seqlen + qrow] = rowf > 0.f ? mc + __builtin_amdgcn_logf(rowf) : INFINITY;
  });
}

// W[bh][p][c] = sum over the rows i of query block p of
// exp2(ylog[bh][c][i] - ylse2[bh][i]).  A workgroup of eight waves takes
// eight consecutive query blocks of one head, one per wave; the waves walk
// the key blocks in the same order, so for each key block the workgroup
// reads one contiguous run of 8 x block rows (4 KB at block 128).  Each wave
// reads its block's rows with one lane per row, BATCH key blocks at a time
// with all their loads in flight together, sums them over the wave in a
// fixed order, and stores 64 masses together.
constexpr int kReduceWaves = 8;
__global__ __launch_bounds__(64 * kReduceWaves) void single_pass_reduce_kernel(AttnParams a) {
  const int bh = blockIdx.y;
  const int L = a.seqlen, nkb = a.nkb;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int p = blockIdx.x * kReduceWaves + wave;
  if (p >= nkb) return;
  const int r0 = p * a.block;
  const int nr = L - r0 < a.block ? L - r0 : a.block;     // rows of this query block
  const bool v0 = lane < nr, v1 = lane + 64 < nr;         // this lane's rows r0 + lane, r0 + lane + 64
  const float* l2 = a.ylse2 + (size_t)bh * L + r0;
  const float m0 = v0 ? l2[lane] : 0.f, m1 = v1 ? l2[lane + 64] : 0.f;
  const float* y = a.ylog + (size_t)bh * nkb * L + r0 + lane;
  constexpr int BATCH = 16;                               // key blocks whose loads are in flight together
  for (int cg = 0; cg < nkb; cg += 64) {
    const int n = nkb - cg < 64 ? nkb - cg : 64;
    float w_mine = 0.f;                                   // lane j keeps block cg + j
    for (int j0 = 0; j0 < n; j0 += BATCH) {
      float y0[BATCH], y1[BATCH];
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const float* yc = y + (size_t)(cg + (j0 + u < n ? j0 + u : n - 1)) * L;
        y0[u] = v0 ? yc[0] : -INFINITY;
        y1[u] = v1 ? yc[64] : -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const float w = wave_sum(fast_exp2(y0[u] - m0) + fast_exp2(y1[u] - m1));
        w_mine = lane == j0 + u ? w : w_mine;
      }
    }
    if (lane < n) a.wmass[((size_t)bh * nkb + p) * nkb + cg + lane] = w_mine;
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
  // 256 query rows per workgroup (eight waves of 32 rows): every K/V tile
  // brought into LDS serves twice the rows of a 128-row workgroup.
  a.row_ptr = nullptr;
  a.col_idx = nullptr;
  a.nqt = (a.seqlen + 255) / 256;
  a.n_items = a.nqt * a.batch_heads;
  a.n_wg = a.n_items;
  if (a.claim != nullptr) {
    // A quarter more workgroups than items: the XCDs that run ahead take the
    // items the others have not reached; surplus workgroups find every queue
    // empty and exit.  The counters are cleared by a kernel (not a memset),
    // so the pair of launches can be captured in a graph.
    a.n_wg = a.n_items + (a.n_items + 3) / 4;
    hipLaunchKernelGGL(claim_reset_kernel, dim3(1), dim3(64), 0, st, a.claim);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (D == 64) return launch_attn<64, 8, false>(a, st);
  return launch_attn<128, 8, false>(a, st);
}

// Work items of block-sparse attention: with a workspace, the first nine
// tenths (rounded down to a multiple of 8) in the static order and the rest
// claimed from the per-XCD queues, with half as many extra workgroups as
// queued items (a fast XCD takes up to that many more than its share).
static hipError_t plan_sparse_items(AttnParams& a, hipStream_t st) {
  a.n_items = a.nqt * a.batch_heads;
  a.n_static = a.n_items;
  a.n_wg = a.n_items;
  if (a.claim == nullptr) return hipSuccess;
  a.n_static = (int)((int64_t)a.n_items * 9 / 10) / 8 * 8;
  a.n_wg = a.n_items + (a.n_items - a.n_static) / 2;
  hipLaunchKernelGGL(claim_reset_kernel, dim3(1), dim3(64), 0, st, a.claim);
  return hipGetLastError();
}

hipError_t launch_sparse(AttnParams a, int D, hipStream_t st) {
  if (a.block == 64) {
    // One workgroup per pair of query blocks (128 rows); text ranges in pairs.
    a.nqt = (a.nkb + 1) / 2;
    if (a.tq1 > a.tq0) {
      a.tq0 = a.tq0 / 2;
      a.tq1 = (a.tq1 + 1) / 2;
      if (a.tq1 - a.tq0 >= a.nqt) a.tq0 = a.tq1 = 0;
    }
    const hipError_t e = plan_sparse_items(a, st);
    if (e != hipSuccess) return e;
    if (D == 64) hipLaunchKernelGGL((attn_sparse_pair_kernel<64, 4>), dim3(a.n_wg), dim3(256), 0, st, a);
    else hipLaunchKernelGGL((attn_sparse_pair_kernel<128, 4>), dim3(a.n_wg), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  // One workgroup per query block of 128 (four waves).
  a.nqt = a.nkb;
  const hipError_t e = plan_sparse_items(a, st);
  if (e != hipSuccess) return e;
  if (D == 64) return launch_attn<64, 4, true>(a, st);
  return launch_attn<128, 4, true>(a, st);
}

template <int D, int QB, int NW>
static hipError_t launch_mass_t(MassParams a, hipStream_t st) {
  a.n_items = (a.nkb + QB - 1) / QB * a.batch_heads;
  a.n_wg = a.n_items;
  if (a.claim != nullptr) {                  // as in launch_dense
    a.n_wg = a.n_items + (a.n_items + 3) / 4;
    hipLaunchKernelGGL(claim_reset_kernel, dim3(1), dim3(64), 0, st, a.claim);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((block_mass_kernel<D, QB, NW>), dim3(a.n_wg), dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_fused_search(AttnParams a, MassParams m, int D, hipStream_t st) {
  // Work items as in launch_dense: (head, 256-row query tile), which is also
  // the mass pass's (head, group of 256 / block query blocks).
  a.row_ptr = nullptr;
  a.col_idx = nullptr;
  a.nqt = (a.seqlen + 255) / 256;
  a.n_items = a.nqt * a.batch_heads;
  a.n_wg = a.n_items;
  if (a.claim != nullptr) {
    a.n_wg = a.n_items + (a.n_items + 3) / 4;
    hipLaunchKernelGGL(claim_reset_kernel, dim3(1), dim3(64), 0, st, a.claim);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  m.claim = nullptr;
  m.n_items = a.n_items;
  m.n_wg = a.n_wg;
  if (a.block == 64) {
    if (D == 64) hipLaunchKernelGGL((fused_search_kernel<64, 4>), dim3(a.n_wg), dim3(512), 0, st, a, m);
    else hipLaunchKernelGGL((fused_search_kernel<128, 4>), dim3(a.n_wg), dim3(512), 0, st, a, m);
  } else {
    if (D == 64) hipLaunchKernelGGL((fused_search_kernel<64, 2>), dim3(a.n_wg), dim3(512), 0, st, a, m);
    else hipLaunchKernelGGL((fused_search_kernel<128, 2>), dim3(a.n_wg), dim3(512), 0, st, a, m);
  }
  return hipGetLastError();
}

hipError_t launch_single_pass_search(AttnParams a, int D, hipStream_t st) {
  // Work items as in launch_dense: (head, 256-row query tile), two query
  // blocks of 128 or four of 64.
  a.row_ptr = nullptr;
  a.col_idx = nullptr;
  a.nqt = (a.seqlen + 255) / 256;
  a.n_items = a.nqt * a.batch_heads;
  a.n_wg = a.n_items;
  if (a.claim != nullptr) {
    a.n_wg = a.n_items + (a.n_items + 3) / 4;
    hipLaunchKernelGGL(claim_reset_kernel, dim3(1), dim3(64), 0, st, a.claim);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (D == 64) hipLaunchKernelGGL((single_pass_search_kernel<64>), dim3(a.n_wg), dim3(512), 0, st, a);
  else hipLaunchKernelGGL((single_pass_search_kernel<128>), dim3(a.n_wg), dim3(512), 0, st, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(single_pass_reduce_kernel, dim3((a.nkb + kReduceWaves - 1) / kReduceWaves, a.batch_heads),
                     dim3(64 * kReduceWaves), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_block_mass(MassParams a, int D, hipStream_t st) {
  // 256 query rows per workgroup: four query blocks of 64 or two of 128.
  if (a.block == 64) {
    if (D == 64) return launch_mass_t<64, 4, 8>(a, st);
    return launch_mass_t<128, 4, 8>(a, st);
  }
  if (D == 64) return launch_mass_t<64, 2, 8>(a, st);
  return launch_mass_t<128, 2, 8>(a, st);
}

}  // namespace adaspa
