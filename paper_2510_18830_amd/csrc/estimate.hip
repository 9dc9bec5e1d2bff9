// Vertical-slash pattern estimation on one GPU (Algorithm 1; Section 4.1).
//
// For each (batch, query head) the last L <= 64 query rows n attend causally
// to the whole sequence: z = scale q_n . k_m for m <= n, P = softmax over m.
//   v_score[m]     = sum_n P[n, m]            (column / vertical scores)
//   s_score[delta] = sum_n P[n, n - delta]    (diagonal / slash scores)
// followed by an exact top-k of each (ties to the lower index, ascending
// output).  The softmax needs each row's normaliser before any column or
// diagonal sum, so K is streamed twice:
//   pass1    per (head, 1024-key chunk): S^T = K Q^T on MFMA, per-row running
//            max and sum of exp2 -> chunk partials
//   combine  per head: log2-sum-exp of the chunk partials for the 64 rows
//   pass2    per (head, chunk): S = Q K^T on MFMA (lane = key), P = exp2(S - lse);
//            column sums reduce within a lane and its partner lane; the 64x64
//            P tile goes to LDS and 127 threads sum its diagonals (sheared
//            read), giving per-tile diagonal partials
//   diag     s_score[64 D + e] = tile(D)[e] + tile(D + 1)[e - 64], in this order
//   topk     radix select of the k-th largest fp32 bit pattern (scores are
//            >= 0, so bit patterns order like values) and an ordered
//            compaction: all entries above it, then the lowest-index ties.
//            With the top-p budget (score_cover of Algorithm 1) a radix select
//            on mass comes first: the same 8-bit digits, each bin carrying
//            its count and its summed mass, finds the value t at which the
//            descending cumulative mass reaches p of the list's total, and k
//            follows from the count and mass above t.
// The last 64 query rows form the last 64-row block exactly (N % 64 == 0), so
// tile j (keys 64 j .. 64 j + 63) holds offsets delta = 64 (nb - 1 - j) + r - c
// for in-block row r and key c.
#include "common.h"
#include "kernels.h"
#include "trace.h"
#include "tiles.h"

namespace msparse {

namespace {

constexpr int kThreads = 128;
constexpr int kChunkTiles = 16;   // 1024 keys per workgroup
constexpr int kMaxGroupWaves = 8;  // query heads per round of the K passes (two waves each)
constexpr float kLog2e = 1.4426950408889634f;

struct EstLayout {
    size_t part_max, part_sum, row_lse, bnd_part, sel_cnt, sel_mass, sel_gt, sel_eq, sel_state, bytes;
};

constexpr int kSliceLen = 16384;   // scores per selection slice
struct SelState {
    uint32_t prefix, mask;   // decided high bits of the selected threshold
    uint32_t krem;           // count select: entries still to take from the prefix group
    uint32_t above;          // entries strictly above the prefix group
    uint64_t rem;            // mass select: mass still to reach (2^-40 units)
    uint32_t k;              // the budget (entries written)
    uint32_t mode;           // kModeMass, kModeCount or kModeDone
};
constexpr uint32_t kModeMass = 1, kModeCount = 2, kModeDone = 3;

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

EstLayout est_layout(int64_t BH, int32_t N) {
    const int64_t nb = N / kBlock;
    const int64_t nchunk = (nb + kChunkTiles - 1) / kChunkTiles;
    EstLayout L{};
    size_t off = 0;
    L.part_max = off;
    off = align256(off + size_t(BH) * nchunk * kBlock * 4);
    L.part_sum = off;
    off = align256(off + size_t(BH) * nchunk * kBlock * 4);
    L.row_lse = off;
    off = align256(off + size_t(BH) * kBlock * 4);
    L.bnd_part = off;
    off = align256(off + size_t(BH) * nchunk * kBlock * 4);
    const int64_t NL = 2 * BH, ns = (N + kSliceLen - 1) / kSliceLen;
    L.sel_cnt = off;
    off = align256(off + size_t(NL) * ns * 256 * 4);
    L.sel_mass = off;
    off = align256(off + size_t(NL) * ns * 256 * 8);
    L.sel_gt = off;
    off = align256(off + size_t(NL) * ns * 8);
    L.sel_eq = off;
    off = align256(off + size_t(NL) * ns * 8);
    L.sel_state = off;
    off = align256(off + size_t(NL) * sizeof(SelState));
    L.bytes = off;
    return L;
}

// ---------------------------------------------------------------- passes over K
// One workgroup per (batch, KV head, chunk of kChunkTiles key tiles) and
// 2 NH waves: waves 2 w and 2 w + 1 serve query rows 0-31 and 32-63 of the
// query heads w, w + NH, ... of the KV group (one round per NH heads), so each
// K tile is read from memory once per group and staged once (direct
// global->LDS loads, double buffer) for all of its heads.  A wave holds its
// 32 query rows as one MFMA operand (qreg); a 64-key tile is two 32-key halves.

// (batch x KV head, chunk) of workgroup t: XCD-chunked, chunks of one KV head
// adjacent.
__device__ __forceinline__ void group_chunk_of(int64_t t, int BK, int nchunk, int& bk, int& chunk) {
    const int64_t u = xcd_chunk(t, int64_t(BK) * nchunk);
    bk = int(u / nchunk);
    chunk = int(u % nchunk);
}

template <int D>
__device__ __forceinline__ void load_qlast(const EstArgs& a, int bh, int rb, int lane, u32x4* qreg) {
    const int h = lane >> 5, l32 = lane & 31;
    const uint16_t* qp = a.q + (int64_t(bh) * a.N + a.N - kBlock + 32 * rb + l32) * D;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) qreg[s] = *reinterpret_cast<const u32x4*>(qp + 16 * s + 8 * h);
}

// pass 1: per-row (max, sum exp2) of the chunk's keys, log2 domain.
// S^T = K Q^T puts one query row per lane (keys in the accumulator).
template <int D, int NH>
__global__ void __launch_bounds__(128 * NH) est_stats_kernel(EstArgs a) {
    constexpr int KD = D / 16;
    constexpr int KE = DmaTile<D, kRowPad>::kElems;
    constexpr int NW = 2 * NH;
    __shared__ uint16_t kt0[KE], kt1[KE];
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), rb = w & 1;
    const int nb = a.N / kBlock, G = a.Hq / a.Hkv;
    int bk, chunk;
    group_chunk_of(blockIdx.x, a.B * a.Hkv, a.nchunk, bk, chunk);
    const int b = bk / a.Hkv, g = bk % a.Hkv;
    const uint16_t* __restrict__ kp = a.k + int64_t(bk) * a.N * D;
    const int j0 = chunk * kChunkTiles, j1 = min(nb, j0 + kChunkTiles);
    const float c2 = a.scale * kLog2e;
    const int row = 32 * rb + l32;
    for (int r0 = 0; r0 < G; r0 += NH) {
        const bool act = r0 + (w >> 1) < G;
        const int bh = b * a.Hq + g * G + (act ? r0 + (w >> 1) : 0);
        u32x4 qreg[KD];
        load_qlast<D>(a, bh, rb, lane, qreg);
        float m = -INFINITY, l = 0.f;
        dma_rows<D, kRowPad, NW>(kt0, kp, ContiguousRows{int64_t(j0) * kBlock}, w, lane);
        wait_vmem();
        __syncthreads();
        for (int j = j0; j < j1; ++j) {
            const uint16_t* cur = ((j - j0) & 1) ? kt1 : kt0;
            if (j + 1 < j1)
                dma_rows<D, kRowPad, NW>(((j - j0) & 1) ? kt0 : kt1, kp, ContiguousRows{int64_t(j + 1) * kBlock}, w,
                                         lane);
            if (act) {
                f32x16 acc[2] = {f32x16{}, f32x16{}};
#pragma unroll
                for (int s = 0; s < KD; ++s)
#pragma unroll
                    for (int kh = 0; kh < 2; ++kh)
                        acc[kh] = mfma32(dma_read16<D, kRowPad>(cur, 32 * kh + l32, h + 2 * s), qreg[s], acc[kh]);
                if (j == nb - 1) {   // keys after the row are masked (causal), only in the last tile
                    keep_branch();
#pragma unroll
                    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            if (32 * kh + 8 * (i >> 2) + 4 * h + (i & 3) > row) acc[kh][i] = -INFINITY;
                }
                float mx = -INFINITY;
#pragma unroll
                for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, acc[kh][i]);
                const float mn = fmaxf(m, mx * c2);
                if (mn != -INFINITY) {
                    float sum = 0.f;
#pragma unroll
                    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                        for (int i = 0; i < 16; ++i) sum += fast_exp2(__builtin_fmaf(acc[kh][i], c2, -mn));
                    l = (m == -INFINITY ? 0.f : l * fast_exp2(m - mn)) + sum;
                    m = mn;
                }
            }
            wait_vmem();
            __syncthreads();
        }
        if (act) {   // the lane pair l, l ^ 32 holds one row
            const float mo = __shfl_xor(m, 32), lo = __shfl_xor(l, 32);
            const float mm = fmaxf(m, mo);
            const float ll = (m == -INFINITY ? 0.f : l * fast_exp2(m - mm)) + (mo == -INFINITY ? 0.f : lo * fast_exp2(mo - mm));
            if (h == 0) {
                const int64_t o = (int64_t(bh) * a.nchunk + chunk) * kBlock + row;
                a.part_max[o] = mm;
                a.part_sum[o] = ll;
            }
        }
    }
}

// One workgroup per (head, 16 rows): 64 threads per row combine the chunk
// partials in a fixed order (per-thread strided runs, then a fixed tree).
constexpr int kCombineRows = 16, kCombineSplit = 64;
__global__ void __launch_bounds__(kCombineRows * kCombineSplit) est_combine_kernel(EstArgs a) {
    __shared__ float pm_s[kCombineRows][kCombineSplit], ps_s[kCombineRows][kCombineSplit];
    const int bh = blockIdx.x / (kBlock / kCombineRows);
    const int rr = threadIdx.x / kCombineSplit, j = threadIdx.x % kCombineSplit;
    const int r = (blockIdx.x % (kBlock / kCombineRows)) * kCombineRows + rr;
    float M = -INFINITY;
    for (int c = j; c < a.nchunk; c += kCombineSplit)
        M = fmaxf(M, a.part_max[(int64_t(bh) * a.nchunk + c) * kBlock + r]);
    float S = 0.f;
    for (int c = j; c < a.nchunk; c += kCombineSplit) {
        const int64_t o = (int64_t(bh) * a.nchunk + c) * kBlock + r;
        const float pm = a.part_max[o];
        if (pm != -INFINITY) S += a.part_sum[o] * fast_exp2(pm - M);
    }
    pm_s[rr][j] = M;
    ps_s[rr][j] = S;
    __syncthreads();
    if (j == 0) {
        float MM = -INFINITY;
        for (int t = 0; t < kCombineSplit; ++t) MM = fmaxf(MM, pm_s[rr][t]);
        float SS = 0.f;
        for (int t = 0; t < kCombineSplit; ++t)
            if (pm_s[rr][t] != -INFINITY) SS += ps_s[rr][t] * fast_exp2(pm_s[rr][t] - MM);
        a.row_lse[bh * kBlock + r] = MM + fast_log2(SS);
    }
}

// Orders the LDS accesses of one wave around a wave-private scratch region.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// pass 2: P = exp2(S - lse) per tile (S = Q K^T, one key per lane), the
// vertical scores (column sums over the 64 rows) and the slash scores.
// Diagonal sums: each 32x32 block (rb, kh) of P goes to the wave's LDS
// scratch; lane e (< 63) sums the block's diagonal r - c = e - 31, which is
// diagonal t = 32 (rb - kh) + e + 32 of the tile (t = r - c + 63 over the
// tile's rows r and keys c).  The two waves of a head leave their column and
// diagonal partials in LDS; after a barrier the row-0 wave adds them in a
// fixed order and writes the scores.  The slash scores are
//   s_score[64 D + e] = T_j[e + 63] + T_{j-1}[e - 1]   (D = nb - 1 - j)
// since the tile j holds offsets delta = 64 (nb - 1 - j) + r - c.  The lower
// part T_{j-1}[e - 1] of a chunk's first tile comes from the previous chunk,
// which leaves it in bnd_part; est_bound_kernel adds it.
template <int D, int NH>
__global__ void __launch_bounds__(128 * NH) est_scores_kernel(EstArgs a) {
    constexpr int KD = D / 16;
    constexpr int KE = DmaTile<D, kRowPad>::kElems;
    constexpr int NW = 2 * NH;
    constexpr int SS = 33;   // scratch row stride (floats)
    __shared__ uint16_t kt0[KE], kt1[KE];
    __shared__ float scr[NW][32 * SS];
    // per head: column partials [rb][64], diagonal partials A, B0, B1, C [64],
    // the previous tile's diagonals 0..63, and the row lse of the head (log2)
    __shared__ float colp[NH][2][kBlock], diagp[NH][4][kBlock], tprev[NH][kBlock];
    __shared__ __attribute__((aligned(16))) float lrow[NH][kBlock];
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), rb = w & 1, hw = w >> 1;
    const int nb = a.N / kBlock, G = a.Hq / a.Hkv;
    int bk, chunk;
    group_chunk_of(blockIdx.x, a.B * a.Hkv, a.nchunk, bk, chunk);
    const int b = bk / a.Hkv, g = bk % a.Hkv;
    const uint16_t* __restrict__ kp = a.k + int64_t(bk) * a.N * D;
    const int j0 = chunk * kChunkTiles, j1 = min(nb, j0 + kChunkTiles);
    const float c2 = a.scale * kLog2e;
    float* sc = scr[w];
    const int e = lane;
    for (int r0 = 0; r0 < G; r0 += NH) {
        const bool act = r0 + hw < G;
        const int bh = b * a.Hq + g * G + (act ? r0 + hw : 0);
        u32x4 qreg[KD];
        load_qlast<D>(a, bh, rb, lane, qreg);
        // rows before the last L contribute nothing
        if (rb == 0) lrow[hw][lane] = lane >= kBlock - a.L ? a.row_lse[bh * kBlock + lane] : INFINITY;
        float* vs = a.v_score + int64_t(bh) * a.N;
        float* ss = a.s_score + int64_t(bh) * a.N;
        dma_rows<D, kRowPad, NW>(kt0, kp, ContiguousRows{int64_t(j0) * kBlock}, w, lane);
        wait_vmem();
        __syncthreads();
        for (int j = j0; j < j1; ++j) {
            const uint16_t* cur = ((j - j0) & 1) ? kt1 : kt0;
            if (j + 1 < j1)
                dma_rows<D, kRowPad, NW>(((j - j0) & 1) ? kt0 : kt1, kp, ContiguousRows{int64_t(j + 1) * kBlock}, w,
                                         lane);
            if (act) {
                const bool last = j == nb - 1;
#pragma unroll
                for (int kh = 0; kh < 2; ++kh) {
                    f32x16 acc = f32x16{};
#pragma unroll
                    for (int s = 0; s < KD; ++s)
                        acc = mfma32(qreg[s], dma_read16<D, kRowPad>(cur, 32 * kh + l32, h + 2 * s), acc);
                    // accumulator element i covers row 32 rb + 8 (i/4) + 4 h + i%4, key 32 kh + l32
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const f32x4 l4 = *reinterpret_cast<const f32x4*>(&lrow[hw][32 * rb + 8 * q4 + 4 * h]);
#pragma unroll
                        for (int e4 = 0; e4 < 4; ++e4)
                            acc[4 * q4 + e4] = fast_exp2(__builtin_fmaf(acc[4 * q4 + e4], c2, -l4[e4]));
                    }
                    if (last) {   // causal mask of the last tile: key > row
                        keep_branch();
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            if (32 * kh + l32 > 32 * rb + 8 * (i >> 2) + 4 * h + (i & 3)) acc[i] = 0.f;
                    }
                    // element (r, c) of the 32 x 32 block goes to scratch row r,
                    // column (c - r) mod 32: column m then holds diagonal r - c = -m
                    // in rows r < 32 - m and diagonal 32 - m in the rows below
                    float cs = 0.f;
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int r = 8 * (i >> 2) + 4 * h + (i & 3);
                        cs += acc[i];
                        sc[r * SS + ((l32 - r) & 31)] = acc[i];
                    }
                    cs = half_swap_sum(cs);
                    if (h == 0) colp[hw][rb][32 * kh + l32] = cs;
                    wave_lds_sync();
                    // lane (h, m) sums rows 16 h .. 16 h + 15 of column m
                    float upper = 0.f, lower = 0.f;
#pragma unroll
                    for (int k = 0; k < 16; ++k) {
                        const int r = 16 * h + k;
                        const float v = sc[r * SS + l32];
                        const bool up = r < 32 - l32;
                        upper += up ? v : 0.f;
                        lower += up ? 0.f : v;
                    }
                    upper = half_swap_sum(upper);
                    lower = half_swap_sum(lower);
                    // diagonal r - c = e - 31 of the block: e = 31 - m from the upper
                    // rows, e = 63 - m from the rest (e = 63 does not exist: 0)
                    // block kind: rb < kh -> A (t = e), rb == kh -> B (t = e + 32), rb > kh -> C (t = e + 64)
                    float* dpk = diagp[hw][rb < kh ? 0 : (rb > kh ? 3 : 1 + rb)];
                    if (h == 0) {
                        dpk[31 - l32] = upper;
                        dpk[63 - l32] = l32 == 0 ? 0.f : lower;
                    }
                    wave_lds_sync();
                }
            }
            __syncthreads();
            if (act && rb == 0) {
                // vertical scores: rows 0-31 + rows 32-63
                vs[int64_t(j) * kBlock + e] = colp[hw][0][e] + colp[hw][1][e];
                // tile diagonals: tlo = T[e] (e < 64), thi = T[64 + e] (e < 63)
                const float* dp = &diagp[hw][0][0];
                const float tlo = dp[e] + (e >= 32 ? dp[kBlock + e - 32] + dp[2 * kBlock + e - 32] : 0.f);
                const float thi = (e < 32 ? dp[kBlock + e + 32] + dp[2 * kBlock + e + 32] : 0.f) + dp[3 * kBlock + e];
                sc[e] = tlo;
                sc[kBlock + e] = thi;
                wave_lds_sync();
                // s_score of block-diagonal D = nb - 1 - j, offset e: T_j[e + 63] + T_{j-1}[e - 1]
                const float up = e == 0 ? sc[63] : sc[kBlock + e - 1];
                const float low = (e >= 1 && j > j0) ? tprev[hw][e - 1] : 0.f;
                ss[int64_t(nb - 1 - j) * kBlock + e] = (e >= 1 && j > j0) ? up + low : up;
                wave_lds_sync();
                tprev[hw][e] = tlo;
                wave_lds_sync();
            }
            wait_vmem();
            __syncthreads();
        }
        // the lower part of the chunk's last tile belongs to the next chunk's first block-diagonal
        if (act && rb == 0 && j1 < nb)
            a.bnd_part[(int64_t(bh) * a.nchunk + chunk) * kBlock + lane] = lane >= 1 ? tprev[hw][lane - 1] : 0.f;
        __syncthreads();
    }
}

// s_score of the first block-diagonal of every chunk after the first: add the
// lower part that the previous chunk left (up + low, as inside a chunk).
__global__ void __launch_bounds__(256) est_bound_kernel(EstArgs a) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t per = int64_t(a.nchunk - 1) * kBlock;   // chunks 1 .. nchunk - 1
    if (i >= int64_t(a.B) * a.Hq * per) return;
    const int64_t bh = i / per;
    const int c = int((i % per) / kBlock) + 1, e = int(i % kBlock);
    if (e == 0) return;
    const int nb = a.N / kBlock;
    const int j0 = c * kChunkTiles;
    const int64_t o = int64_t(bh) * a.N + int64_t(nb - 1 - j0) * kBlock + e;
    a.s_score[o] = a.s_score[o] + a.bnd_part[(bh * a.nchunk + c - 1) * kBlock + e];
}

// ---------------------------------------------------------------- top-k / top-p
// Selection over the 2 B Hq score lists (vertical lists first), each cut into
// slices of kSliceLen scores: per digit (8 bits, high first) a histogram pass
// over every (list, slice) writes per-slice bin counts (and masses), and a
// select pass per list sums them in slice order and narrows the prefix.  With
// a top-p fraction, four mass digits find the threshold score t at which the
// descending cumulative mass reaches p of the total; then four count digits
// (skipped by lists already decided) find the k-th largest for fixed budgets
// or for capped ones.  Two compaction passes write all entries above the
// threshold and the lowest-index ties, in index order.  Scores are >= 0, so
// fp32 bit patterns order like values.
constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / 64;
// Histograms are private per wave (stride 257 words, so the copies sit on
// different banks): the scores of a list share few exponents, and one shared
// histogram would serialise nearly every atomic on the same bins.  Scores are
// read 4 at a time (16-byte loads, N % 64 == 0), several loads in flight per
// thread.
constexpr int kHistStride = 257;

// Adds 1 to bin `bin` of the wave's histogram for every lane with `on`.  The
// lanes sharing the first pending lane's bin are counted with a ballot and
// added by one lane, up to 4 rounds (the scores of a list share few
// exponents, so most digits fall in a handful of bins); the rest add singly.
__device__ __forceinline__ void hist_add(uint32_t* wh, uint32_t bin, bool on) {
    const int lane = threadIdx.x & 63;
    bool pending = on;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const uint64_t pm = __ballot(pending);
        if (pm == 0) return;
        const int first = __builtin_ctzll(pm);
        const uint32_t lb = uint32_t(__shfl(int(bin), first));
        const bool same = pending && bin == lb;
        const uint64_t sm = __ballot(same);
        if (lane == first) atomicAdd(&wh[lb], uint32_t(__popcll(sm)));
        pending = pending && !same;
    }
    if (pending) atomicAdd(&wh[bin], 1u);
}
// Masses in fixed point: a score x (0 <= x <= L <= 64) counts floor(x 2^40), so
// every sum of masses is an exact integer (below 2^47) whatever the order of
// the additions, and the budget is deterministic.
__device__ __forceinline__ uint64_t mass_fx(uint32_t bits) {
    return uint64_t(double(__uint_as_float(bits)) * 1099511627776.0);
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// hist_add with a mass: the lanes of one ballot group add their summed mass.
__device__ __forceinline__ void hist_add_mass(uint32_t* wh, uint64_t* wm, uint32_t bin, uint64_t mass, bool on) {
    const int lane = threadIdx.x & 63;
    bool pending = on;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const uint64_t pm = __ballot(pending);
        if (pm == 0) return;
        const int first = __builtin_ctzll(pm);
        const uint32_t lb = uint32_t(__shfl(int(bin), first));
        const bool same = pending && bin == lb;
        const uint64_t sm = __ballot(same);
        const uint64_t ms = wave_sum_u64(same ? mass : 0ull);
        if (lane == first) {
            atomicAdd(&wh[lb], uint32_t(__popcll(sm)));
            atomicAdd(reinterpret_cast<unsigned long long*>(&wm[lb]), (unsigned long long)ms);
        }
        pending = pending && !same;
    }
    if (pending) {
        atomicAdd(&wh[bin], 1u);
        atomicAdd(reinterpret_cast<unsigned long long*>(&wm[bin]), (unsigned long long)mass);
    }
}

__device__ __forceinline__ SelState* sel_state(const EstArgs& a) { return reinterpret_cast<SelState*>(a.sel_state); }

__global__ void __launch_bounds__(256) sel_init_kernel(EstArgs a) {
    const int NL = 2 * a.B * a.Hq;
    const int l = blockIdx.x * 256 + threadIdx.x;
    if (l >= NL) return;
    const bool is_v = l < a.B * a.Hq;
    SelState st{};
    st.mode = (is_v ? a.p_v : a.p_s) > 0.0 ? kModeMass : kModeCount;
    st.krem = uint32_t(is_v ? a.k_v : a.k_s);
    st.k = st.krem;
    sel_state(a)[l] = st;
}

// one (list, slice) per workgroup: histogram of digit `shift` over the scores
// that match the list's prefix
template <bool MASS>
__global__ void __launch_bounds__(kSelThreads) sel_hist_kernel(EstArgs a, int shift) {
    __shared__ uint32_t whist[kSelWaves * kHistStride];
    __shared__ uint64_t wmass[MASS ? kSelWaves * 256 : 1];
    const int list = blockIdx.x / a.nslice, slice = blockIdx.x % a.nslice;
    const SelState st = sel_state(a)[list];
    if (st.mode != (MASS ? kModeMass : kModeCount)) return;
    const int BH = a.B * a.Hq;
    const float* sc = (list < BH ? a.v_score + int64_t(list) * a.N : a.s_score + int64_t(list - BH) * a.N);
    const u32x4* sc4 = reinterpret_cast<const u32x4*>(sc);
    const int tid = threadIdx.x, wv = tid >> 6;
    for (int i = tid; i < kSelWaves * kHistStride; i += kSelThreads) whist[i] = 0;
    if (MASS)
        for (int i = tid; i < kSelWaves * 256; i += kSelThreads) wmass[i] = 0;
    __syncthreads();
    uint32_t* wh = whist + wv * kHistStride;
    const int lo4 = slice * (kSliceLen / 4), hi4 = min(a.N / 4, lo4 + kSliceLen / 4);
    for (int i0 = lo4 + tid; i0 < hi4; i0 += 4 * kSelThreads) {
        u32x4 x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = i0 + u * kSelThreads;
            x[u] = i < hi4 ? sc4[i] : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const bool in = i0 + u * kSelThreads < hi4;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool on = in && (x[u][e] & st.mask) == st.prefix;
                const uint32_t bin = (x[u][e] >> shift) & 255u;
                if (MASS) hist_add_mass(wh, wmass + wv * 256, bin, mass_fx(x[u][e]), on);
                else hist_add(wh, bin, on);
            }
        }
    }
    __syncthreads();
    const int64_t o = (int64_t(list) * a.nslice + slice) * 256;
    for (int b = tid; b < 256; b += kSelThreads) {
        uint32_t c = 0;
        uint64_t m = 0;
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) {
            c += whist[w * kHistStride + b];
            if (MASS) m += wmass[w * 256 + b];
        }
        a.sel_cnt[o + b] = c;
        if (MASS) a.sel_mass[o + b] = m;
    }
}

// one list per workgroup: sum the slices' bins (fixed order) and narrow the prefix
template <bool MASS>
__global__ void __launch_bounds__(256) sel_pick_kernel(EstArgs a, int shift) {
    __shared__ uint32_t hc[256];
    __shared__ uint64_t hm[MASS ? 256 : 1];
    const int list = blockIdx.x;
    SelState* stp = sel_state(a) + list;
    const SelState st0 = *stp;
    if (st0.mode != (MASS ? kModeMass : kModeCount)) return;
    const int b = threadIdx.x;
    uint32_t c = 0;
    uint64_t m = 0;
    // slices in groups of 8: the group's loads are all in flight at once
    constexpr int U = 8;
    for (int sl0 = 0; sl0 < a.nslice; sl0 += U) {
        uint32_t cu[U];
        uint64_t mu[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int sl = sl0 + u;
            const int64_t o = (int64_t(list) * a.nslice + (sl < a.nslice ? sl : 0)) * 256 + b;
            cu[u] = sl < a.nslice ? a.sel_cnt[o] : 0u;
            mu[u] = MASS && sl < a.nslice ? a.sel_mass[o] : 0u;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            c += cu[u];
            m += mu[u];
        }
    }
    hc[b] = c;
    if (MASS) hm[b] = m;
    __syncthreads();
    if (b != 0) return;
    SelState st = st0;
    const int BH = a.B * a.Hq;
    const bool is_v = list < BH;
    const uint32_t cap = uint32_t(is_v ? a.k_v : a.k_s);
    if (MASS) {
        if (shift == 24) {
            // every score matches the empty prefix: the bins hold the total mass
            uint64_t total = 0;
            for (int bb = 0; bb < 256; ++bb) total += hm[bb];
            if (total == 0) {   // no mass at all: one entry reaches p of it
                st.mode = kModeCount;
                st.krem = 1;
                st.k = 1;
                *stp = st;
                return;
            }
            st.rem = uint64_t(ceil((is_v ? a.p_v : a.p_s) * double(total)));
        }
        // the prefix group holds at least rem (> 0) of mass, so some bin is taken
        uint64_t run = 0;
        uint32_t runc = 0;
        int bsel = 0;
        for (int bb = 255; bb >= 0; --bb) {
            if (run + hm[bb] >= st.rem) {
                bsel = bb;
                break;
            }
            run += hm[bb];
            runc += hc[bb];
        }
        st.prefix |= uint32_t(bsel) << shift;
        st.mask |= 255u << shift;
        st.rem -= run;
        st.above += runc;
        if (shift == 0) {
            // t = prefix; every score equal to t adds mass_fx(t)
            const uint64_t qt = mass_fx(st.prefix);
            const uint64_t ties = qt ? (st.rem + qt - 1) / qt : uint64_t(hc[bsel]);
            const uint64_t k = uint64_t(st.above) + min<uint64_t>(ties, hc[bsel]);
            if (k <= cap) {
                st.k = uint32_t(k);
                st.krem = uint32_t(k) - st.above;
                st.mode = kModeDone;
            } else {   // capped: the count select finds the cap-th largest
                st.k = cap;
                st.krem = cap;
                st.prefix = 0;
                st.mask = 0;
                st.above = 0;
                st.mode = kModeCount;
            }
        }
    } else {
        uint32_t run = 0;
        int bsel = 0;
        for (int bb = 255; bb >= 0; --bb) {
            if (run + hc[bb] >= st.krem) {
                bsel = bb;
                break;
            }
            run += hc[bb];
        }
        st.prefix |= uint32_t(bsel) << shift;
        st.mask |= 255u << shift;
        st.krem -= run;
        st.above += run;
        if (shift == 0) st.mode = kModeDone;
    }
    *stp = st;
}

// per (list, slice): entries above the threshold and ties with it
__global__ void __launch_bounds__(kSelThreads) sel_count_kernel(EstArgs a) {
    __shared__ int64_t wgt[kSelWaves], weq[kSelWaves];
    const int list = blockIdx.x / a.nslice, slice = blockIdx.x % a.nslice;
    const SelState st = sel_state(a)[list];
    const int BH = a.B * a.Hq;
    const uint32_t* sc = reinterpret_cast<const uint32_t*>(list < BH ? a.v_score + int64_t(list) * a.N
                                                                      : a.s_score + int64_t(list - BH) * a.N);
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int lo = slice * kSliceLen, hi = min(a.N, lo + kSliceLen);
    int64_t gt = 0, eq = 0;
    for (int i0 = lo + wv * 64; i0 < hi; i0 += kSelThreads) {
        const int i = i0 + lane;
        const uint32_t x = i < hi ? sc[i] : 0u;
        gt += __popcll(__ballot(i < hi && x > st.prefix));
        eq += __popcll(__ballot(i < hi && x == st.prefix));
    }
    if (lane == 0) {
        wgt[wv] = gt;
        weq[wv] = eq;
    }
    __syncthreads();
    if (tid == 0) {
        int64_t g = 0, e = 0;
        for (int w = 0; w < kSelWaves; ++w) {
            g += wgt[w];
            e += weq[w];
        }
        a.sel_gt[int64_t(list) * a.nslice + slice] = g;
        a.sel_eq[int64_t(list) * a.nslice + slice] = e;
    }
}

// per (list, slice): write the slice's selected indices at its offset, in
// index order (wave-contiguous sub-slices, ballots for the ranks)
__global__ void __launch_bounds__(kSelThreads) sel_write_kernel(EstArgs a) {
    __shared__ int64_t wgt[kSelWaves], weq[kSelWaves];
    const int list = blockIdx.x / a.nslice, slice = blockIdx.x % a.nslice;
    const SelState st = sel_state(a)[list];
    const int BH = a.B * a.Hq;
    const bool is_v = list < BH;
    const int cap = is_v ? a.k_v : a.k_s;
    const uint32_t* sc = reinterpret_cast<const uint32_t*>(is_v ? a.v_score + int64_t(list) * a.N
                                                                : a.s_score + int64_t(list - BH) * a.N);
    int32_t* out = (is_v ? a.v_idx + int64_t(list) * cap : a.s_idx + int64_t(list - BH) * cap);
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    // slices before this one: entries taken and ties seen
    int64_t off = 0, eq_before = 0;
    for (int sl = 0; sl < slice; ++sl) {
        off += a.sel_gt[int64_t(list) * a.nslice + sl];
        eq_before += a.sel_eq[int64_t(list) * a.nslice + sl];
    }
    off += min<int64_t>(eq_before, st.krem);
    // this slice: wave wv owns [lo + wv C, lo + (wv + 1) C)
    const int lo = slice * kSliceLen, hi = min(a.N, lo + kSliceLen);
    const int C = ((hi - lo + kSelWaves * 64 - 1) / (kSelWaves * 64)) * 64;
    const int wlo = lo + wv * C, whi = min(hi, wlo + C);
    const uint64_t below = (1ull << lane) - 1ull;
    int64_t gt = 0, eq = 0;
    for (int i0 = wlo; i0 < whi; i0 += 64) {
        const int i = i0 + lane;
        const uint32_t x = i < whi ? sc[i] : 0u;
        gt += __popcll(__ballot(i < whi && x > st.prefix));
        eq += __popcll(__ballot(i < whi && x == st.prefix));
    }
    if (lane == 0) {
        wgt[wv] = gt;
        weq[wv] = eq;
    }
    __syncthreads();
    for (int w = 0; w < wv; ++w) {
        off += wgt[w] + min<int64_t>(weq[w], max<int64_t>(0, int64_t(st.krem) - eq_before));
        eq_before += weq[w];
    }
    for (int i0 = wlo; i0 < whi; i0 += 64) {
        const int i = i0 + lane;
        const uint32_t x = i < whi ? sc[i] : 0u;
        const bool e = i < whi && x == st.prefix;
        const uint64_t me = __ballot(e);
        const bool take = (i < whi && x > st.prefix) || (e && eq_before + __popcll(me & below) < int64_t(st.krem));
        const uint64_t mt = __ballot(take);
        if (take) out[off + __popcll(mt & below)] = i;
        off += __popcll(mt);
        eq_before += __popcll(me);
    }
}

// top-p lists: the budget and -1 in the unused slots
__global__ void __launch_bounds__(256) sel_finish_kernel(EstArgs a) {
    const int list = blockIdx.x;
    const SelState st = sel_state(a)[list];
    const int BH = a.B * a.Hq;
    const bool is_v = list < BH;
    const int cap = is_v ? a.k_v : a.k_s;
    int32_t* out = (is_v ? a.v_idx + int64_t(list) * cap : a.s_idx + int64_t(list - BH) * cap);
    for (int i = int(st.k) + threadIdx.x; i < cap; i += 256) out[i] = -1;
    if (threadIdx.x == 0) (is_v ? a.v_cnt + list : a.s_cnt + (list - BH))[0] = int32_t(st.k);
}

hipError_t launch_select(const EstArgs& a, hipStream_t s) {
    const int NL = 2 * a.B * a.Hq;
    const unsigned grid = unsigned(NL * a.nslice);
    const bool topp = a.p_v > 0.0;
    { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_init_kernel, dim3((NL + 255) / 256), dim3(256), 0, s, a); }
    if (topp)
        for (int shift = 24; shift >= 0; shift -= 8) {
            { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_hist_kernel<true>, dim3(grid), dim3(kSelThreads), 0, s, a, shift); }
            { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_pick_kernel<true>, dim3(NL), dim3(256), 0, s, a, shift); }
        }
    for (int shift = 24; shift >= 0; shift -= 8) {
        { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_hist_kernel<false>, dim3(grid), dim3(kSelThreads), 0, s, a, shift); }
        { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_pick_kernel<false>, dim3(NL), dim3(256), 0, s, a, shift); }
    }
    { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_count_kernel, dim3(grid), dim3(kSelThreads), 0, s, a); }
    { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_write_kernel, dim3(grid), dim3(kSelThreads), 0, s, a); }
    if (topp) { TraceScope _t("est_topk", s); hipLaunchKernelGGL(sel_finish_kernel, dim3(NL), dim3(256), 0, s, a); }
    return hipGetLastError();
}

template <int D, int NW>
hipError_t launch_passes(const EstArgs& a, hipStream_t s) {
    const int BH = a.B * a.Hq;
    const unsigned grid = unsigned(a.B * a.Hkv * a.nchunk);
    { TraceScope _t("est_pass1", s); hipLaunchKernelGGL((est_stats_kernel<D, NW>), dim3(grid), dim3(128 * NW), 0, s, a); }
    { TraceScope _t("est_combine", s); hipLaunchKernelGGL(est_combine_kernel, dim3(BH * (kBlock / kCombineRows)), dim3(kCombineRows * kCombineSplit), 0, s, a); }
    { TraceScope _t("est_pass2", s); hipLaunchKernelGGL((est_scores_kernel<D, NW>), dim3(grid), dim3(128 * NW), 0, s, a); }
    if (a.nchunk > 1) {
        const int64_t n = int64_t(BH) * (a.nchunk - 1) * kBlock;
        TraceScope _t("est_bound", s);
        hipLaunchKernelGGL(est_bound_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

template <int D>
hipError_t launch_d(const EstArgs& a, hipStream_t s) {
    hipError_t e;
    switch (std::min(a.Hq / a.Hkv, kMaxGroupWaves)) {   // two waves per query head of the KV group
        case 1: e = launch_passes<D, 1>(a, s); break;
        case 2: e = launch_passes<D, 2>(a, s); break;
        case 3: e = launch_passes<D, 3>(a, s); break;
        case 4: e = launch_passes<D, 4>(a, s); break;
        case 5: e = launch_passes<D, 5>(a, s); break;
        case 6: e = launch_passes<D, 6>(a, s); break;
        case 7: e = launch_passes<D, 7>(a, s); break;
        default: e = launch_passes<D, 8>(a, s); break;
    }
    if (e != hipSuccess) return e;
    return launch_select(a, s);
}

}  // namespace

size_t est_workspace_bytes(int32_t B, int32_t Hq, int32_t N, int32_t L) {
    (void)L;
    return est_layout(int64_t(B) * Hq, N).bytes;
}

void est_carve(EstArgs& a, char* base) {
    const EstLayout L = est_layout(int64_t(a.B) * a.Hq, a.N);
    a.nchunk = (a.N / kBlock + kChunkTiles - 1) / kChunkTiles;
    a.part_max = reinterpret_cast<float*>(base + L.part_max);
    a.part_sum = reinterpret_cast<float*>(base + L.part_sum);
    a.row_lse = reinterpret_cast<float*>(base + L.row_lse);
    a.bnd_part = reinterpret_cast<float*>(base + L.bnd_part);
    a.nslice = (a.N + kSliceLen - 1) / kSliceLen;
    a.sel_cnt = reinterpret_cast<uint32_t*>(base + L.sel_cnt);
    a.sel_mass = reinterpret_cast<uint64_t*>(base + L.sel_mass);
    a.sel_gt = reinterpret_cast<int64_t*>(base + L.sel_gt);
    a.sel_eq = reinterpret_cast<int64_t*>(base + L.sel_eq);
    a.sel_state = base + L.sel_state;
}

hipError_t launch_estimate(const EstArgs& a, hipStream_t s) {
    return a.d == 128 ? launch_d<128>(a, s) : launch_d<64>(a, s);
}

}  // namespace msparse
