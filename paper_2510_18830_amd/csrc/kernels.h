// Host-side launchers of the gfx950 kernels (internal to libmsparse).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/msparse.h"

namespace msparse {

// ---------------------------------------------------------------- index build
struct IndexArgs {
    const int32_t* v_idx;  // [BH, k_v] global token positions
    const int32_t* s_idx;  // [BH, k_s] global slash offsets
    int32_t BH, k_v, k_s;
    int32_t nqb, nkb;      // local query / key blocks
    int32_t nb;            // global blocks
    int32_t world, rank, shard, layout;
    // workspace carve-up
    uint32_t* vbits;       // [BH, vwords]
    int32_t vwords;
    int32_t* vlist;        // [BH, k_v] unique ascending verticals
    int32_t* vcnt;         // [BH]
    int32_t* dlist;        // [BH, nb] ascending block-diagonals
    int32_t* dcnt;         // [BH]
    uint32_t* dbits;       // [BH, dwords]
    int32_t dwords;
    int32_t* dpre;         // [BH, dwords + 1] selected block-diagonals in the words before each word
    int32_t* cumv;         // [BH, nb + 1] verticals in the (global) blocks before each block
    int32_t* drun;         // [BH] R: block-diagonals 0 .. R-1 are all selected, R is not
    int64_t* cnt_blk;      // [BH*nqb]
    int64_t* cnt_col;      // [BH*nqb]
    int64_t* cnt_kblk;     // [BH*nkb]
    int64_t* cnt_vcol;     // [BH]
    int64_t* scan_sums;    // [4, scan_stride] per-block sums of the scan
    int64_t scan_stride;
    // scanned offsets (n + 1 entries each)
    int64_t* blk_ptr;
    int64_t* col_ptr;
    int64_t* kblk_ptr;
    int64_t* vcol_ptr;
    // outputs (fill only)
    int32_t* blk_idx;
    int64_t blk_cap;
    int32_t* col_idx;
    int64_t col_cap;
    int32_t* kblk_idx;
    int32_t* vcol_idx;
    int64_t vcol_cap;
    uint32_t* diag_bits_out;
    int32_t* q_blk_global;
    int32_t* k_blk_global;
    int32_t* overflow;
};
hipError_t launch_index_prep(const IndexArgs& a, hipStream_t s);
// the prefix scans of the index counts: blocks of kScanEntriesPerBlock entries,
// at most kScanEntriesPerBlock blocks per array
constexpr int kScanEntriesPerBlock = 4096;
// worker x shard tiles / columns of a ring of `world` workers (prep first)
constexpr int32_t kMaxRingWorld = 4096;
hipError_t launch_ring_work(const IndexArgs& a, int32_t world, int32_t layout, int64_t* tiles, int64_t* cols,
                            hipStream_t s);
hipError_t launch_index_count(const IndexArgs& a, hipStream_t s);
hipError_t launch_index_scan(const IndexArgs& a, hipStream_t s);
hipError_t launch_index_fill(const IndexArgs& a, hipStream_t s);
// *a.overflow = 1 (one thread; the lists of the index are not filled)
hipError_t launch_index_mark_overflow(const IndexArgs& a, hipStream_t s);

// ---------------------------------------------------------------- attention
struct AttnArgs {
    const uint16_t* q;     // bf16 [B,Hq,Nq,d]
    const uint16_t* k;     // bf16 [B,Hkv,Nk,d]
    const uint16_t* v;
    uint16_t* v16;         // fp16 copies of the second-GEMM operands (workspace):
    uint16_t* k16;         //   V (fwd), K (dQ), Q and s dO (dK / dV)
    uint16_t* q16;
    uint16_t* g16;
    const uint16_t* o;     // forward output (bwd)
    const uint16_t* dout;  // bf16 [B,Hq,Nq,d] (bwd)
    uint16_t* out;         // bf16 [B,Hq,Nq,d] (fwd)
    float* out_f32;        // optional fp32 copy of out (fwd)
    const float* o_f32;    // optional fp32 forward output for Delta (bwd)
    uint32_t* dmax;        // bwd workspace: max |dO| as fp32 bits
    uint32_t* qkvmax;      // workspace: max |Q|, |K|, |V| as fp32 bits (the fwd uses [2])
    float* lse;            // fwd output / bwd input
    float* draw;           // bwd workspace [B,Hq,Nq]: Delta = dO . O (query-side, reusable)
    float* delta;          // bwd workspace [B,Hq,Nq]: t * s * Delta, t = dz_scale() (per call, row prep)
    float* lse2;           // bwd workspace [B,Hq,Nq]: lse * log2(e) (+inf for a row without keys)
    float* dq;
    float* dk;
    float* dv;
    float* dk_col;         // bwd workspace [col_slots, 64, d]: per-item column partials
    float* dv_col;
    int64_t vcol_cap;
    // bwd column-pass work list (workspace, written by the plan kernel)
    int32_t* col_choff;    // [B*Hq + 1] first chunk of each head; last = chunk count
    int64_t* col_e0;       // [col_chunk_cap] first vertical entry of each chunk
    int32_t* col_head;     // [col_chunk_cap] head (b * Hq + h) of each chunk
    int32_t* col_qlo;      // [col_chunk_cap] first local query block that may see the chunk
    int32_t* col_item;     // [col_chunk_cap + 1] first item of each chunk; last = item count
    int32_t* col_span;     // [1] query blocks per item
    int64_t col_chunk_cap;
    int64_t col_budget;    // items the span is chosen for
    int64_t col_slots;     // item capacity (grid of the column kernel)
    int32_t dq_accumulate;
    int32_t reuse_qrows;   // the workspace already holds the Q-side data (a later ring step)
    int32_t merge_acc;     // fwd: out_f32 / lse hold a running (o, lse) that the result is merged into
    int32_t B, Hq, Hkv, Nq, Nk, d;
    int32_t nqb, nkb;
    float scale;
    const int64_t* blk_ptr;
    const int32_t* blk_idx;
    const int64_t* col_ptr;
    const int32_t* col_idx;
    const int64_t* kblk_ptr;
    const int32_t* kblk_idx;
    const int64_t* vcol_ptr;
    const int32_t* vcol_idx;
    const uint32_t* diag_bits;
    int32_t dwords;
    const int32_t* q_blk_global;
    const int32_t* k_blk_global;
    // set by an index build that ran out of capacity (may be NULL): every
    // kernel that walks the lists then returns before reading them
    const int32_t* overflow;
};
hipError_t launch_attn_fwd(const AttnArgs& a, hipStream_t s);
// *maxbits = max(*maxbits, max |src|) as fp32 bits, n bf16 elements (n a
// multiple of 8)
hipError_t launch_absmax(const uint16_t* src, int64_t n, uint32_t* maxbits, hipStream_t s);
// dst = fp16(src * mul) for n bf16 elements (n a multiple of 8); mul = 1 when
// maxbits is NULL, else the power of two pow2_scale_to<exp>(maxbits) (exp 4
// for dO, kOperandExp for Q, K, V)
hipError_t launch_to_f16(const uint16_t* src, uint16_t* dst, int64_t n, const uint32_t* maxbits, int exp,
                         hipStream_t s);
hipError_t launch_attn_bwd(const AttnArgs& a, hipStream_t s);
// Backward column pass: a chunk is 64 consecutive entries of one head's
// vertical list; its candidate query blocks (a suffix of the local blocks) are
// split into items of `span` blocks, one workgroup each.  span is the smallest
// value >= kColMinSpan that keeps the item count within the budget.
constexpr int kColItems = 2048;
constexpr int kColMinSpan = 16;
struct ColPlanSizes {
    int64_t chunk_cap;  // bound on the chunk count: sum over heads of ceil(n_h / 64)
    int64_t budget;
    int64_t slots;      // bound on the item count: budget + chunk_cap
};
inline ColPlanSizes col_plan_sizes(int64_t bh, int64_t vcol_cap, int64_t nqb) {
    ColPlanSizes z;
    z.chunk_cap = (vcol_cap + 63) / 64 + bh;
    const int64_t fine = z.chunk_cap * ((nqb + kColMinSpan - 1) / kColMinSpan);
    z.budget = fine < kColItems ? fine : kColItems;
    z.slots = z.budget + z.chunk_cap;
    return z;
}

struct MergeArgs {
    const float* o_part;
    const float* lse_part;
    float* o_acc;
    float* lse_acc;
    uint16_t* out;
    int32_t first;
    int64_t rows;  // B*Hq*Nq
    int32_t d;
};
hipError_t launch_merge(const MergeArgs& a, hipStream_t s);

// ---------------------------------------------------------------- estimation
struct EstArgs {
    const uint16_t* q;  // bf16 [B,Hq,N,d]
    const uint16_t* k;  // bf16 [B,Hkv,N,d]
    int32_t B, Hq, Hkv, N, d, L, k_v, k_s;
    float scale;
    float* v_score;     // [B*Hq, N]
    float* s_score;     // [B*Hq, N]
    int32_t* v_idx;     // [B*Hq, k_v]
    int32_t* s_idx;     // [B*Hq, k_s]
    // top-p budget (p_v > 0): k_v / k_s are the caps, the budgets go to
    // v_cnt / s_cnt [B*Hq] and the unused slots of v_idx / s_idx are set to -1
    double p_v, p_s;
    int32_t* v_cnt;
    int32_t* s_cnt;
    // workspace (est_carve)
    float* part_max;    // [B*Hq, nchunk, 64]
    float* part_sum;    // [B*Hq, nchunk, 64]
    float* row_lse;     // [B*Hq, 64] (log2 domain)
    float* bnd_part;    // [B*Hq, nchunk, 64]: lower diagonal part of each chunk's last tile
    int32_t nchunk;
    // selection (top-k / top-p) over 2 B Hq lists of N scores cut into nslice
    // slices: per-slice histograms and compaction counts, per-list state
    int32_t nslice;
    uint32_t* sel_cnt;  // [2 BH, nslice, 256]
    uint64_t* sel_mass; // [2 BH, nslice, 256]
    int64_t* sel_gt;    // [2 BH, nslice]
    int64_t* sel_eq;    // [2 BH, nslice]
    void* sel_state;    // [2 BH] selection state
};
size_t est_workspace_bytes(int32_t B, int32_t Hq, int32_t N, int32_t L);
void est_carve(EstArgs& a, char* base);
hipError_t launch_estimate(const EstArgs& a, hipStream_t s);

}  // namespace msparse
