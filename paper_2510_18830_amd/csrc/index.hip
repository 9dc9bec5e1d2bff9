// Sparse index construction on the GPU (Section 4.1 (ii); convert_index of
// Algorithms 1 and 2).
//
// Each selected slash offset delta is executed as the 64 x 64 block-diagonals
// floor(delta/64) and ceil(delta/64) (the set D); query block i gets the key
// blocks i - x (x in D, x <= i) and the verticals v <= 64 i + 63 that lie in a
// block-diagonal outside D.  A ring step keeps only the keys of its KV shard,
// in that shard's local numbering.
//
// Four launches, all deterministic (no atomics decide an output position):
//   prep  one workgroup per head: vertical bitmap -> unique ascending list,
//         slash offsets -> D bitset -> ascending list, shard vertical counts;
//   count one wavefront per (head, query block) and per (head, key block);
//   scan  exclusive prefix sums of the counts (one workgroup per array);
//   fill  the count pass again, writing entries in order via wave ballots.
// The ring workload matrix (msparse_ring_work) reuses prep and counts, per
// (head, worker, chunk of the worker's query blocks), the tiles and columns
// that fall into each worker's KV shard.
#include "common.h"
#include "kernels.h"
#include "trace.h"

namespace msparse {

namespace {

constexpr int kPrepThreads = 1024;
constexpr int kItemWaves = 4;  // wavefronts per workgroup in count / fill

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ uint64_t lanes_below() { return (1ull << lane_id()) - 1ull; }

// Exclusive prefix sum over a 1024-thread workgroup.  `tmp` holds 16 ints.
__device__ int block_exclusive_scan(int v, int* tmp, int* total) {
    const int lane = lane_id(), wid = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) tmp[wid] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int w = 0; w < kPrepThreads / 64; ++w) {
            int t = tmp[w];
            tmp[w] = run;
            run += t;
        }
        tmp[16] = run;
    }
    __syncthreads();
    int res = tmp[wid] + x - v;
    *total = tmp[16];
    __syncthreads();
    return res;
}

__global__ void __launch_bounds__(kPrepThreads) index_prep_kernel(IndexArgs a) {
    __shared__ int tmp[17];
    extern __shared__ uint32_t dsh[];  // D bitset, dwords words
    const int bh = blockIdx.x;
    const int tid = threadIdx.x;
    const Layout L{a.world, a.nb, a.layout};
    const int64_t Ng = int64_t(a.nb) * kBlock;

    // the overflow flag starts at 0 for this build (a kernel store, not a memset,
    // so that the call can be captured in a graph); the fill pass may set it
    if (bh == 0 && tid == 0 && a.overflow) *a.overflow = 0;
    // ---- verticals: bitmap (dedupes and sorts), then ordered compaction
    uint32_t* vb = a.vbits + int64_t(bh) * a.vwords;
    for (int w = tid; w < a.vwords; w += kPrepThreads) vb[w] = 0u;
    for (int w = tid; w < a.dwords; w += kPrepThreads) dsh[w] = 0u;
    __threadfence();
    __syncthreads();
    const int32_t* vi = a.v_idx + int64_t(bh) * a.k_v;
    for (int j = tid; j < a.k_v; j += kPrepThreads) {
        int32_t v = vi[j];
        if (v >= 0 && v < Ng) atomicOr(&vb[v >> 5], 1u << (v & 31));
    }
    const int32_t* si = a.s_idx + int64_t(bh) * a.k_s;
    for (int j = tid; j < a.k_s; j += kPrepThreads) {
        int32_t dl = si[j];
        if (dl < 0 || dl >= Ng) continue;
        int32_t lo = dl / kBlock, hi = (dl + kBlock - 1) / kBlock;
        atomicOr(&dsh[lo >> 5], 1u << (lo & 31));
        if (hi < a.nb) atomicOr(&dsh[hi >> 5], 1u << (hi & 31));
    }
    __threadfence();
    __syncthreads();

    // each thread owns a contiguous run of bitmap words
    {
        const int per = (a.vwords + kPrepThreads - 1) / kPrepThreads;
        const int w0 = tid * per, w1 = min(a.vwords, w0 + per);
        int cnt = 0, own = 0;
        for (int w = w0; w < w1; ++w) {
            uint32_t bits = __atomic_load_n(&vb[w], __ATOMIC_RELAXED);
            cnt += __popc(bits);
            for (uint32_t b = bits; b; b &= b - 1) {
                int32_t v = (w << 5) + __ffs(b) - 1;
                own += (L.owner(v / kBlock) == a.shard);
            }
        }
        int total = 0;
        int pos = block_exclusive_scan(cnt, tmp, &total);
        int32_t* out = a.vlist + int64_t(bh) * a.k_v;
        for (int w = w0; w < w1; ++w) {
            uint32_t bits = __atomic_load_n(&vb[w], __ATOMIC_RELAXED);
            for (uint32_t b = bits; b; b &= b - 1) out[pos++] = (w << 5) + __ffs(b) - 1;
        }
        int owned = 0;
        block_exclusive_scan(own, tmp, &owned);
        if (tid == 0) {
            a.vcnt[bh] = total;
            a.cnt_vcol[bh] = owned;
        }
    }
    // ---- block-diagonals: bitset copy and ascending list
    {
        uint32_t* db = a.dbits + int64_t(bh) * a.dwords;
        for (int w = tid; w < a.dwords; w += kPrepThreads) {
            db[w] = dsh[w];
            if (a.diag_bits_out) a.diag_bits_out[int64_t(bh) * a.dwords + w] = dsh[w];
        }
        const int per = (a.dwords + kPrepThreads - 1) / kPrepThreads;
        const int w0 = tid * per, w1 = min(a.dwords, w0 + per);
        int cnt = 0;
        for (int w = w0; w < w1; ++w) cnt += __popc(dsh[w]);
        int total = 0;
        int pos = block_exclusive_scan(cnt, tmp, &total);
        int32_t* out = a.dlist + int64_t(bh) * a.nb;
        for (int w = w0; w < w1; ++w)
            for (uint32_t b = dsh[w]; b; b &= b - 1) out[pos++] = (w << 5) + __ffs(b) - 1;
        if (tid == 0) a.dcnt[bh] = total;
        // prefix counts per word (dpre) and the run of selected diagonals from 0
        int32_t* dp = a.dpre + int64_t(bh) * (a.dwords + 1);
        int run = 0;
        for (int w = w0; w < w1; ++w) {
            dp[w] = pos - cnt + run;
            run += __popc(dsh[w]);
        }
        if (tid == 0) {
            dp[a.dwords] = total;
            tmp[16] = a.nb;
        }
        __syncthreads();
        for (int w = tid; w < a.dwords; w += kPrepThreads)
            if (dsh[w] != 0xffffffffu) atomicMin(&tmp[16], (w << 5) + __ffs(~dsh[w]) - 1);
        __syncthreads();
        if (tid == 0) a.drun[bh] = min(tmp[16], a.nb);
        __syncthreads();
    }
    // ---- verticals per global block, as prefix counts (cumv)
    {
        const int per = (a.nb + kPrepThreads - 1) / kPrepThreads;
        const int j0 = tid * per, j1 = min(a.nb, j0 + per);
        int cnt = 0;
        for (int j = j0; j < j1; ++j)
            cnt += __popc(__atomic_load_n(&vb[2 * j], __ATOMIC_RELAXED)) +
                   __popc(__atomic_load_n(&vb[2 * j + 1], __ATOMIC_RELAXED));
        int total = 0;
        int pos = block_exclusive_scan(cnt, tmp, &total);
        int32_t* cv = a.cumv + int64_t(bh) * (a.nb + 1);
        for (int j = j0; j < j1; ++j) {
            cv[j] = pos;
            pos += __popc(__atomic_load_n(&vb[2 * j], __ATOMIC_RELAXED)) +
                   __popc(__atomic_load_n(&vb[2 * j + 1], __ATOMIC_RELAXED));
        }
        if (tid == 0) cv[a.nb] = total;
    }
    if (bh == 0) {
        if (a.q_blk_global)
            for (int l = tid; l < a.nqb; l += kPrepThreads) a.q_blk_global[l] = L.global(a.rank, l);
        if (a.k_blk_global)
            for (int l = tid; l < a.nkb; l += kPrepThreads) a.k_blk_global[l] = L.global(a.shard, l);
    }
}

__device__ __forceinline__ bool dbit(const uint32_t* db, int32_t x) { return (db[x >> 5] >> (x & 31)) & 1u; }

// Number of selected block-diagonals below x (0 <= x <= nb) from the per-word
// prefix counts.
__device__ __forceinline__ int32_t diag_below(const int32_t* dp, const uint32_t* db, int32_t x) {
    const int w = x >> 5, b = x & 31;
    return dp[w] + (b ? __popc(db[w] & ((1u << b) - 1u)) : 0);
}

// Sum over the lanes of a wavefront.
__device__ __forceinline__ int64_t wave_sum64(int64_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// Whole-sequence index (one worker): closed forms from the prefix counts.
// Query block i has the key blocks i - x for the diag_below(i + 1) selected x
// <= i, and as columns the verticals of blocks j <= i - R (blocks i - R + 1 ..
// i lie on the selected diagonals 0 .. R-1) minus those whose diagonal i - j
// is selected; key block k has the query blocks k + x, x < nb - k.
template <bool FILL>
__device__ void whole_query_item(const IndexArgs& a, int64_t item, int bh, int32_t i, int lane) {
    const int32_t* dl = a.dlist + int64_t(bh) * a.nb;
    const uint32_t* db = a.dbits + int64_t(bh) * a.dwords;
    const int32_t* dp = a.dpre + int64_t(bh) * (a.dwords + 1);
    const int32_t* cv = a.cumv + int64_t(bh) * (a.nb + 1);
    const int32_t nblk = diag_below(dp, db, i + 1);
    const int32_t R = min(a.drun[bh], i + 1);
    const int32_t nscan = cv[i - R + 1];   // verticals of blocks 0 .. i - R
    if (!FILL) {
        int64_t far = 0;   // verticals of blocks i - x, x selected, R <= x <= i
        for (int j = R + lane; j < nblk; j += 64) {
            const int32_t jb = i - dl[j];
            far += cv[jb + 1] - cv[jb];
        }
        far = wave_sum64(far);
        if (lane == 0) {
            a.cnt_blk[item] = nblk;
            a.cnt_col[item] = nscan - far;
        }
        return;
    }
    const int64_t bbase = a.blk_ptr[item];
    if (a.blk_ptr[item + 1] > a.blk_cap) {
        if (lane == 0 && a.overflow) atomicOr(a.overflow, 1);
    } else {
        for (int j = lane; j < nblk; j += 64) a.blk_idx[bbase + j] = i - dl[nblk - 1 - j];
    }
    const int64_t cbase = a.col_ptr[item];
    if (a.col_ptr[item + 1] > a.col_cap) {
        if (lane == 0 && a.overflow) atomicOr(a.overflow, 1);
        return;
    }
    const int32_t* vl = a.vlist + int64_t(bh) * a.k_v;
    int64_t n = 0;
    for (int c0 = 0; c0 < nscan; c0 += 64) {
        const int j = c0 + lane;
        int32_t v = 0;
        bool pred = false;
        if (j < nscan) {
            v = vl[j];
            pred = !dbit(db, i - v / kBlock);
        }
        const uint64_t m = __ballot(pred);
        if (pred) a.col_idx[cbase + n + __popcll(m & lanes_below())] = v;
        n += __popcll(m);
    }
}

template <bool FILL>
__device__ void whole_key_item(const IndexArgs& a, int64_t it, int bh, int32_t k, int lane) {
    const int32_t* dl = a.dlist + int64_t(bh) * a.nb;
    const uint32_t* db = a.dbits + int64_t(bh) * a.dwords;
    const int32_t* dp = a.dpre + int64_t(bh) * (a.dwords + 1);
    const int32_t cnt = diag_below(dp, db, a.nb - k);
    if (!FILL) {
        if (lane == 0) a.cnt_kblk[it] = cnt;
        return;
    }
    if (a.kblk_ptr[it + 1] > a.blk_cap) {
        if (lane == 0 && a.overflow) atomicOr(a.overflow, 1);
        return;
    }
    const int64_t base = a.kblk_ptr[it];
    for (int j = lane; j < cnt; j += 64) a.kblk_idx[base + j] = k + dl[j];
}

// One wavefront walks the lists of one item.  FILL = false counts, FILL = true
// writes the entries at the scanned offsets.
template <bool FILL>
__global__ void __launch_bounds__(64 * kItemWaves) index_items_kernel(IndexArgs a) {
    int64_t item = int64_t(blockIdx.x) * kItemWaves + (threadIdx.x >> 6);
    const int lane = lane_id();
    const Layout L{a.world, a.nb, a.layout};
    const int64_t nq_items = int64_t(a.BH) * a.nqb;
    const int64_t nk_items = int64_t(a.BH) * a.nkb;
    if (!FILL && a.world == 1 && item >= nq_items) {
        // whole-sequence key-block counts are one lookup each: 64 per wave
        const int64_t it = (item - nq_items) * 64 + lane;
        if (it < nk_items) {
            const int bh = int(it / a.nkb);
            const int32_t k = int32_t(it % a.nkb);
            a.cnt_kblk[it] = diag_below(a.dpre + int64_t(bh) * (a.dwords + 1), a.dbits + int64_t(bh) * a.dwords,
                                        a.nb - k);
        }
        return;
    }

    if (item < nq_items) {
        const int bh = int(item / a.nqb);
        const int lq = int(item % a.nqb);
        if (a.world == 1) {
            whole_query_item<FILL>(a, item, bh, lq, lane);
            return;
        }
        const int32_t qg = L.global(a.rank, lq);
        const int32_t* dl = a.dlist + int64_t(bh) * a.nb;
        const int dc = a.dcnt[bh];
        const uint32_t* db = a.dbits + int64_t(bh) * a.dwords;
        // ---- key blocks qg - x, x in D, ascending key block = descending x
        int64_t base = FILL ? a.blk_ptr[item] : 0;
        bool ok = true;
        if (FILL) {
            if (a.blk_ptr[item + 1] > a.blk_cap) {
                ok = false;
                if (lane == 0 && a.overflow) atomicOr(a.overflow, 1);
            }
        }
        int64_t n = 0;
        for (int c0 = 0; c0 < dc; c0 += 64) {
            const int j = dc - 1 - (c0 + lane);
            bool pred = false;
            int32_t kg = 0;
            if (j >= 0) {
                const int32_t x = dl[j];
                kg = qg - x;
                pred = (x <= qg) && (L.owner(kg) == a.shard);
            }
            const uint64_t m = __ballot(pred);
            if (FILL && ok && pred) a.blk_idx[base + n + __popcll(m & lanes_below())] = L.local(kg);
            n += __popcll(m);
        }
        if (!FILL && lane == 0) a.cnt_blk[item] = n;
        // ---- columns: verticals v <= 64 qg + 63 outside the selected diagonals
        const int32_t* vl = a.vlist + int64_t(bh) * a.k_v;
        const int vc = a.vcnt[bh];
        const int32_t limit = qg * kBlock + kBlock - 1;
        base = FILL ? a.col_ptr[item] : 0;
        ok = true;
        if (FILL) {
            if (a.col_ptr[item + 1] > a.col_cap) {
                ok = false;
                if (lane == 0 && a.overflow) atomicOr(a.overflow, 1);
            }
        }
        n = 0;
        for (int c0 = 0; c0 < vc; c0 += 64) {
            if (vl[c0] > limit) break;  // list is ascending
            const int j = c0 + lane;
            bool pred = false;
            int32_t v = 0;
            if (j < vc) {
                v = vl[j];
                const int32_t vb = v / kBlock;
                pred = (v <= limit) && !dbit(db, qg - vb) && (L.owner(vb) == a.shard);
            }
            const uint64_t m = __ballot(pred);
            if (FILL && ok && pred)
                a.col_idx[base + n + __popcll(m & lanes_below())] = L.local(v / kBlock) * kBlock + v % kBlock;
            n += __popcll(m);
        }
        if (!FILL && lane == 0) a.cnt_col[item] = n;
        return;
    }
    if (item < nq_items + nk_items) {
        // ---- transposed block lists: query blocks kg + x, x in D, ascending
        const int64_t it = item - nq_items;
        const int bh = int(it / a.nkb);
        const int lk = int(it % a.nkb);
        if (a.world == 1) {
            whole_key_item<FILL>(a, it, bh, lk, lane);
            return;
        }
        const int32_t kg = L.global(a.shard, lk);
        const int32_t* dl = a.dlist + int64_t(bh) * a.nb;
        const int dc = a.dcnt[bh];
        int64_t base = FILL ? a.kblk_ptr[it] : 0;
        bool ok = true;
        if (FILL && a.kblk_ptr[it + 1] > a.blk_cap) {
            ok = false;
            if (lane == 0 && a.overflow) atomicOr(a.overflow, 1);
        }
        int64_t n = 0;
        for (int c0 = 0; c0 < dc; c0 += 64) {
            const int j = c0 + lane;
            bool pred = false;
            int32_t qg = 0;
            if (j < dc) {
                qg = kg + dl[j];
                pred = (qg < a.nb) && (L.owner(qg) == a.rank);
            }
            const uint64_t m = __ballot(pred);
            if (FILL && ok && pred) a.kblk_idx[base + n + __popcll(m & lanes_below())] = L.local(qg);
            n += __popcll(m);
        }
        if (!FILL && lane == 0) a.cnt_kblk[it] = n;
        return;
    }
    if (FILL && item < nq_items + nk_items + a.BH) {
        // ---- this shard's verticals in local coordinates
        const int bh = int(item - nq_items - nk_items);
        const int32_t* vl = a.vlist + int64_t(bh) * a.k_v;
        const int vc = a.vcnt[bh];
        const int64_t base = a.vcol_ptr[bh];
        if (a.vcol_ptr[bh + 1] > a.vcol_cap) {
            if (lane == 0 && a.overflow) atomicOr(a.overflow, 1);
            return;
        }
        int64_t n = 0;
        for (int c0 = 0; c0 < vc; c0 += 64) {
            const int j = c0 + lane;
            bool pred = false;
            int32_t v = 0;
            if (j < vc) {
                v = vl[j];
                pred = L.owner(v / kBlock) == a.shard;
            }
            const uint64_t m = __ballot(pred);
            if (pred) a.vcol_idx[base + n + __popcll(m & lanes_below())] = L.local(v / kBlock) * kBlock + v % kBlock;
            n += __popcll(m);
        }
    }
}

// dst[0] = 0, dst[i + 1] = cnt[0] + ... + cnt[i] for the four count arrays
// (gridDim.y selects the array): per-block sums of kScanBlock entries, one
// workgroup scans the block sums (kept in the workspace), then every block
// scans its own entries from its offset.  Loads are coalesced and the sums are
// integers, so the result does not depend on the grid.
constexpr int kScanThreads = 256;
constexpr int kScanPer = 16;
constexpr int kScanBlock = kScanThreads * kScanPer;   // 4096 entries per block
static_assert(kScanBlock == kScanEntriesPerBlock, "scan geometry");

__device__ __forceinline__ void scan_array(const IndexArgs& a, int which, const int64_t*& cnt, int64_t*& dst,
                                           int64_t& n) {
    switch (which) {
        case 0: cnt = a.cnt_blk; dst = a.blk_ptr; n = int64_t(a.BH) * a.nqb; break;
        case 1: cnt = a.cnt_col; dst = a.col_ptr; n = int64_t(a.BH) * a.nqb; break;
        case 2: cnt = a.cnt_kblk; dst = a.kblk_ptr; n = int64_t(a.BH) * a.nkb; break;
        default: cnt = a.cnt_vcol; dst = a.vcol_ptr; n = a.BH; break;
    }
}

// exclusive scan of one value per thread over the workgroup; returns the total in *total
__device__ int64_t block_scan64(int64_t v, int64_t* tmp, int64_t* total) {
    const int lane = lane_id(), wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) tmp[wid] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t run = 0;
        for (int w = 0; w < nw; ++w) {
            const int64_t t = tmp[w];
            tmp[w] = run;
            run += t;
        }
        tmp[16] = run;
    }
    __syncthreads();
    const int64_t res = tmp[wid] + x - v;
    *total = tmp[16];
    __syncthreads();
    return res;
}

__global__ void __launch_bounds__(kScanThreads) index_scan_sums_kernel(IndexArgs a) {
    __shared__ int64_t tmp[17];
    const int64_t* cnt;
    int64_t* dst;
    int64_t n;
    scan_array(a, blockIdx.y, cnt, dst, n);
    const int64_t base = int64_t(blockIdx.x) * kScanBlock;
    if (base >= n) return;
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        const int64_t i = base + j * kScanThreads + threadIdx.x;
        if (i < n) s += cnt[i];
    }
    int64_t total = 0;
    block_scan64(s, tmp, &total);
    if (threadIdx.x == 0) a.scan_sums[int64_t(blockIdx.y) * a.scan_stride + blockIdx.x] = total;
}

// one workgroup per array: exclusive scan of the block sums (at most kScanThreads * kScanPer blocks)
__global__ void __launch_bounds__(kScanThreads) index_scan_top_kernel(IndexArgs a) {
    __shared__ int64_t tmp[17];
    const int64_t* cnt;
    int64_t* dst;
    int64_t n;
    scan_array(a, blockIdx.x, cnt, dst, n);
    const int nblk = int((n + kScanBlock - 1) / kScanBlock);
    int64_t* sums = a.scan_sums + int64_t(blockIdx.x) * a.scan_stride;
    // thread t owns sums [t * kScanPer, (t + 1) * kScanPer)
    int64_t v[kScanPer];
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        const int i = threadIdx.x * kScanPer + j;
        v[j] = i < nblk ? sums[i] : 0;
        s += v[j];
    }
    int64_t total = 0;
    int64_t run = block_scan64(s, tmp, &total);
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        const int i = threadIdx.x * kScanPer + j;
        if (i < nblk) sums[i] = run;
        run += v[j];
    }
    if (threadIdx.x == 0) dst[0] = 0;
}

__global__ void __launch_bounds__(kScanThreads) index_scan_fill_kernel(IndexArgs a) {
    __shared__ int64_t tmp[17];
    __shared__ int64_t vals[kScanBlock];
    const int64_t* cnt;
    int64_t* dst;
    int64_t n;
    scan_array(a, blockIdx.y, cnt, dst, n);
    const int64_t base = int64_t(blockIdx.x) * kScanBlock;
    if (base >= n) return;
    // coalesced load into LDS, then thread t scans entries [t * kScanPer, (t + 1) * kScanPer)
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        const int k = j * kScanThreads + threadIdx.x;
        vals[k] = base + k < n ? cnt[base + k] : 0;
    }
    __syncthreads();
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) s += vals[threadIdx.x * kScanPer + j];
    int64_t total = 0;
    int64_t run = block_scan64(s, tmp, &total) + a.scan_sums[int64_t(blockIdx.y) * a.scan_stride + blockIdx.x];
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        const int k = threadIdx.x * kScanPer + j;
        run += vals[k];
        vals[k] = run;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        const int k = j * kScanThreads + threadIdx.x;
        if (base + k < n) dst[base + k + 1] = vals[k];
    }
}

// ---------------------------------------------------------------- ring workload
constexpr int kWorkThreads = 256;
constexpr int kWorkChunk = 64;   // query blocks per workgroup

// Adds 1 to bin `bin` for every lane with `on`: lanes sharing the first pending
// lane's bin are counted with a ballot (zigzag shards are runs of neighbouring
// blocks, so most lanes share a bin), up to four rounds, then single adds.
__device__ __forceinline__ void bin_add(uint32_t* h, int32_t bin, bool on) {
    bool pending = on;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const uint64_t pm = __ballot(pending);
        if (pm == 0) return;
        const int first = __builtin_ctzll(pm);
        const int32_t lb = __shfl(bin, first);
        const bool same = pending && bin == lb;
        const uint64_t sm = __ballot(same);
        if (lane_id() == first) atomicAdd(&h[lb], uint32_t(__popcll(sm)));
        pending = pending && !same;
    }
    if (pending) atomicAdd(&h[bin], 1u);
}

__global__ void __launch_bounds__(256) ring_work_zero_kernel(int64_t* tiles, int64_t* cols, int64_t n) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
        tiles[i] = 0;
        cols[i] = 0;
    }
}

__global__ void __launch_bounds__(kWorkThreads) ring_work_kernel(IndexArgs a, int32_t W, int32_t layout,
                                                                 int64_t* tiles, int64_t* cols) {
    __shared__ uint32_t ht[kMaxRingWorld], hc[kMaxRingWorld];
    const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
    const Layout L{W, a.nb, layout};
    const int per = a.nb / W;                        // query blocks per worker
    const int nchunk = (per + kWorkChunk - 1) / kWorkChunk;
    int item = blockIdx.x;
    const int chunk = item % nchunk;
    item /= nchunk;
    const int r = item % W;
    const int bh = item / W;
    for (int i = tid; i < W; i += kWorkThreads) {
        ht[i] = 0;
        hc[i] = 0;
    }
    __syncthreads();
    const int32_t* dl = a.dlist + int64_t(bh) * a.nb;
    const int dc = a.dcnt[bh];
    const uint32_t* db = a.dbits + int64_t(bh) * a.dwords;
    const int32_t* vl = a.vlist + int64_t(bh) * a.k_v;
    const int vc = a.vcnt[bh];
    const int l1 = min(per, (chunk + 1) * kWorkChunk);
    for (int l = chunk * kWorkChunk + wave; l < l1; l += kWorkThreads / 64) {
        const int32_t i = L.global(r, l);
        // tiles (i, i - x), x in D, x <= i
        for (int c0 = 0; c0 < dc; c0 += 64) {
            const int j = c0 + lane;
            const int32_t x = j < dc ? dl[j] : 0;
            const bool on = j < dc && x <= i;
            bin_add(ht, on ? L.owner(i - x) : 0, on);
        }
        // columns v <= 64 i + 63 whose block-diagonal is not in D
        const int32_t limit = i * kBlock + kBlock - 1;
        for (int c0 = 0; c0 < vc; c0 += 64) {
            if (vl[c0] > limit) break;   // ascending list
            const int j = c0 + lane;
            const int32_t v = j < vc ? vl[j] : 0;
            const bool on = j < vc && v <= limit && !dbit(db, i - v / kBlock);
            bin_add(hc, on ? L.owner(v / kBlock) : 0, on);
        }
    }
    __syncthreads();
    for (int sh = tid; sh < W; sh += kWorkThreads) {
        if (ht[sh]) atomicAdd(reinterpret_cast<unsigned long long*>(tiles + int64_t(r) * W + sh), (unsigned long long)ht[sh]);
        if (hc[sh]) atomicAdd(reinterpret_cast<unsigned long long*>(cols + int64_t(r) * W + sh), (unsigned long long)hc[sh]);
    }
}

}  // namespace

hipError_t launch_ring_work(const IndexArgs& a, int32_t world, int32_t layout, int64_t* tiles, int64_t* cols,
                            hipStream_t s) {
    const int64_t n = int64_t(world) * world;
    {
        TraceScope _t("ring_work_zero", s);
        hipLaunchKernelGGL(ring_work_zero_kernel, dim3(unsigned(std::min<int64_t>((n + 255) / 256, 4096))), dim3(256),
                           0, s, tiles, cols, n);
    }
    const int per = a.nb / world;
    const int64_t grid = int64_t(a.BH) * world * ((per + kWorkChunk - 1) / kWorkChunk);
    {
        TraceScope _t("ring_work", s);
        hipLaunchKernelGGL(ring_work_kernel, dim3(unsigned(grid)), dim3(kWorkThreads), 0, s, a, world, layout, tiles,
                           cols);
    }
    return hipGetLastError();
}

hipError_t launch_index_prep(const IndexArgs& a, hipStream_t s) {
    const size_t shmem = size_t(a.dwords) * sizeof(uint32_t);
    { TraceScope _t("index_prep", s); hipLaunchKernelGGL(index_prep_kernel, dim3(a.BH), dim3(kPrepThreads), shmem, s, a); }
    return hipGetLastError();
}

hipError_t launch_index_count(const IndexArgs& a, hipStream_t s) {
    const int64_t nk = int64_t(a.BH) * a.nkb;
    const int64_t items = int64_t(a.BH) * a.nqb + (a.world == 1 ? (nk + 63) / 64 : nk);
    const int64_t grid = (items + kItemWaves - 1) / kItemWaves;
    { TraceScope _t("index_count", s); hipLaunchKernelGGL(index_items_kernel<false>, dim3(unsigned(grid)), dim3(64 * kItemWaves), 0, s, a); }
    return hipGetLastError();
}

hipError_t launch_index_scan(const IndexArgs& a, hipStream_t s) {
    const int64_t nmax = std::max<int64_t>(int64_t(a.BH) * std::max(a.nqb, a.nkb), a.BH);
    const unsigned nblk = unsigned((nmax + kScanBlock - 1) / kScanBlock);
    { TraceScope _t("index_scan", s); hipLaunchKernelGGL(index_scan_sums_kernel, dim3(nblk, 4), dim3(kScanThreads), 0, s, a); }
    { TraceScope _t("index_scan", s); hipLaunchKernelGGL(index_scan_top_kernel, dim3(4), dim3(kScanThreads), 0, s, a); }
    { TraceScope _t("index_scan", s); hipLaunchKernelGGL(index_scan_fill_kernel, dim3(nblk, 4), dim3(kScanThreads), 0, s, a); }
    return hipGetLastError();
}

__global__ void index_mark_overflow_kernel(int32_t* flag) {
    if (threadIdx.x == 0) *flag = 1;
}

hipError_t launch_index_mark_overflow(const IndexArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(index_mark_overflow_kernel, dim3(1), dim3(64), 0, s, a.overflow);
    return hipGetLastError();
}

hipError_t launch_index_fill(const IndexArgs& a, hipStream_t s) {
    const int64_t items = int64_t(a.BH) * (a.nqb + a.nkb) + a.BH;
    const int64_t grid = (items + kItemWaves - 1) / kItemWaves;
    { TraceScope _t("index_fill", s); hipLaunchKernelGGL(index_items_kernel<true>, dim3(unsigned(grid)), dim3(64 * kItemWaves), 0, s, a); }
    return hipGetLastError();
}

}  // namespace msparse
