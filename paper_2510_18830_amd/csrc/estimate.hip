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
constexpr float kLog2e = 1.4426950408889634f;

struct EstLayout {
    size_t part_max, part_sum, row_lse, diag_part, bytes;
};

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
    L.diag_part = off;
    off = align256(off + size_t(BH) * nb * 128 * 4);
    L.bytes = off;
    return L;
}

template <int D>
struct Pass1Lds {
    uint16_t k[TileLds<D>::kRowElems];
};

// pass 1: per-row (max, sum exp2) over one chunk of keys, log2 domain
template <int D>
__global__ void __launch_bounds__(kThreads) est_pass1_kernel(EstArgs a) {
    constexpr int KD = D / 16;
    __shared__ Pass1Lds<D> sm;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
    const int nb = a.N / kBlock;
    // KV-group-major order, XCD-chunked: the group's heads read each K chunk
    // together from one L2
    int bh, chunk;
    query_tile_of(blockIdx.x, a.B, a.Hq, a.Hkv, a.nchunk, bh, chunk);
    const int b = bh / a.Hq, hq = bh % a.Hq, hk = hq / (a.Hq / a.Hkv);
    const int row = 32 * w + l32;   // in the last block
    const uint16_t* qp = a.q + (int64_t(bh) * a.N + a.N - kBlock + row) * D;
    const uint16_t* kp = a.k + (int64_t(b) * a.Hkv + hk) * int64_t(a.N) * D;
    u32x4 qreg[KD];
#pragma unroll
    for (int s = 0; s < KD; ++s) qreg[s] = *reinterpret_cast<const u32x4*>(qp + 16 * s + 8 * h);
    const float c2 = a.scale * kLog2e;
    float m = -INFINITY, l = 0.f;
    const int j0 = chunk * kChunkTiles, j1 = min(nb, j0 + kChunkTiles);
    for (int j = j0; j < j1; ++j) {
        stage_rows<D, kThreads>(sm.k, kp, ContiguousRows{int64_t(j) * kBlock}, tid);
        __syncthreads();
        f32x16 acc[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            acc[c] = f32x16{};
            const uint16_t* krow = sm.k + (32 * c + l32) * TileLds<D>::kRowStride + 8 * h;
#pragma unroll
            for (int s = 0; s < KD; ++s) acc[c] = mfma32(lds_read16(krow + 16 * s), qreg[s], acc[c]);
        }
        const bool last = j == nb - 1;
        float mx = -INFINITY;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = 32 * c + 8 * (r >> 2) + 4 * h + (r & 3);
                float x = acc[c][r] * c2;
                if (last && key > row) x = -INFINITY;
                acc[c][r] = x;
                mx = fmaxf(mx, x);
            }
        const float mn = fmaxf(m, mx);   // finite: every row sees key 0
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int r = 0; r < 16; ++r) s += fast_exp2(acc[c][r] - mn);
        l = l * fast_exp2(m - mn) + s;
        m = mn;
        __syncthreads();
    }
    // combine the two lane halves (same row)
    const float mo = __shfl_xor(m, 32), lo = __shfl_xor(l, 32);
    const float mm = fmaxf(m, mo);
    const float ll = (m == -INFINITY ? 0.f : l * fast_exp2(m - mm)) + (mo == -INFINITY ? 0.f : lo * fast_exp2(mo - mm));
    if (h == 0) {
        const int64_t o = (int64_t(bh) * a.nchunk + chunk) * kBlock + row;
        a.part_max[o] = mm;
        a.part_sum[o] = ll;
    }
}

// One workgroup per head: thread (r, j) reduces chunks j, j + 16, ... of row
// r; the 16 partials of a row are combined in a fixed order.
constexpr int kCombineSplit = 16;
__global__ void __launch_bounds__(64 * kCombineSplit) est_combine_kernel(EstArgs a) {
    __shared__ float pm_s[kCombineSplit][64], ps_s[kCombineSplit][64];
    const int bh = blockIdx.x, r = threadIdx.x & 63, j = threadIdx.x >> 6;
    float M = -INFINITY;
    for (int c = j; c < a.nchunk; c += kCombineSplit) M = fmaxf(M, a.part_max[(int64_t(bh) * a.nchunk + c) * kBlock + r]);
    float S = 0.f;
    for (int c = j; c < a.nchunk; c += kCombineSplit) {
        const int64_t o = (int64_t(bh) * a.nchunk + c) * kBlock + r;
        const float pm = a.part_max[o];
        if (pm != -INFINITY) S += a.part_sum[o] * fast_exp2(pm - M);
    }
    pm_s[j][r] = M;
    ps_s[j][r] = S;
    __syncthreads();
    if (j == 0) {
        float MM = -INFINITY;
        for (int t = 0; t < kCombineSplit; ++t) MM = fmaxf(MM, pm_s[t][r]);
        float SS = 0.f;
        for (int t = 0; t < kCombineSplit; ++t)
            if (pm_s[t][r] != -INFINITY) SS += ps_s[t][r] * fast_exp2(pm_s[t][r] - MM);
        a.row_lse[bh * kBlock + r] = MM + fast_log2(SS);
    }
}

template <int D>
struct Pass2Lds {
    uint16_t k[TileLds<D>::kRowElems];
    float p[64][65];
    float col[2][64];
};

template <int D>
__global__ void __launch_bounds__(kThreads) est_pass2_kernel(EstArgs a) {
    constexpr int KD = D / 16;
    __shared__ Pass2Lds<D> sm;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
    const int nb = a.N / kBlock;
    int bh, chunk;   // order as in pass 1
    query_tile_of(blockIdx.x, a.B, a.Hq, a.Hkv, a.nchunk, bh, chunk);
    const int b = bh / a.Hq, hq = bh % a.Hq, hk = hq / (a.Hq / a.Hkv);
    // A operand: this wave's 32 query rows
    const uint16_t* qp = a.q + (int64_t(bh) * a.N + a.N - kBlock + 32 * w + l32) * D;
    const uint16_t* kp = a.k + (int64_t(b) * a.Hkv + hk) * int64_t(a.N) * D;
    u32x4 qreg[KD];
#pragma unroll
    for (int s = 0; s < KD; ++s) qreg[s] = *reinterpret_cast<const u32x4*>(qp + 16 * s + 8 * h);
    // accumulator element r covers row 32 w + 8 (r/4) + 4 h + r%4
    float lse2[16];
    bool valid[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int row = 32 * w + 8 * (r >> 2) + 4 * h + (r & 3);
        lse2[r] = a.row_lse[bh * kBlock + row];
        valid[r] = row >= kBlock - a.L;
    }
    const float c2 = a.scale * kLog2e;
    const int j0 = chunk * kChunkTiles, j1 = min(nb, j0 + kChunkTiles);
    for (int j = j0; j < j1; ++j) {
        stage_rows<D, kThreads>(sm.k, kp, ContiguousRows{int64_t(j) * kBlock}, tid);
        __syncthreads();
        const bool last = j == nb - 1;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            f32x16 acc = f32x16{};
            const uint16_t* krow = sm.k + (32 * c + l32) * TileLds<D>::kRowStride + 8 * h;
#pragma unroll
            for (int s = 0; s < KD; ++s) acc = mfma32(qreg[s], lds_read16(krow + 16 * s), acc);
            const int key = 32 * c + l32;
            float cs = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = 32 * w + 8 * (r >> 2) + 4 * h + (r & 3);
                float p = fast_exp2(acc[r] * c2 - lse2[r]);
                if (!valid[r] || (last && key > row)) p = 0.f;
                sm.p[row][key] = p;
                cs += p;
            }
            cs += __shfl_xor(cs, 32);
            if (h == 0) sm.col[w][key] = cs;
        }
        __syncthreads();
        if (tid < 64) a.v_score[int64_t(bh) * a.N + int64_t(j) * kBlock + tid] = sm.col[0][tid] + sm.col[1][tid];
        if (tid < 127) {
            // delta_local = r - c = tid - 63: a fixed 64-step walk, masked at
            // the ends, four accumulators (the reads pipeline; neighbouring
            // threads read neighbouring words)
            const int dl = tid - 63;
            float s4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int r = 0; r < 64; ++r) {
                const int c = r - dl;
                const float v = sm.p[r][c & 63];
                s4[r & 3] += (c >= 0 && c < 64) ? v : 0.f;
            }
            a.diag_part[(int64_t(bh) * nb + j) * 128 + tid] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
        }
        __syncthreads();
    }
}

// s_score[64 D + e] = tile(j = nb-1-D)[e + 63] + tile(j - 1)[e - 1]  (e >= 1)
__global__ void __launch_bounds__(256) est_diag_kernel(EstArgs a) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int nb = a.N / kBlock;
    if (i >= int64_t(a.B) * a.Hq * a.N) return;
    const int64_t bh = i / a.N;
    const int dlt = int(i % a.N);
    const int Dg = dlt / kBlock, e = dlt % kBlock;
    const int j = nb - 1 - Dg;
    float s = a.diag_part[(bh * nb + j) * 128 + e + 63];
    if (e >= 1 && j >= 1) s += a.diag_part[(bh * nb + j - 1) * 128 + e - 1];
    a.s_score[i] = s;
}

// ---------------------------------------------------------------- top-k
constexpr int kTopkThreads = 1024;


// Histograms are private per wave (16 copies, stride 257 words so the copies
// sit on different banks): scores of one list share few exponents, and one
// shared histogram would serialise nearly every atomic on the same bins.
// Scores are read 4 at a time (16-byte loads, N % 64 == 0), several loads in
// flight per thread.
constexpr int kHistStride = 257;
constexpr int kTopkWaves = kTopkThreads / 64;

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

struct TopkLds {
    uint32_t whist[kTopkWaves * kHistStride];
    uint64_t wmass[kTopkWaves * 256];
    uint32_t hist[256];
    uint64_t hmass[256];
    uint64_t wsum[kTopkWaves];
    uint32_t s_prefix, s_krem, s_k, s_above;
    uint64_t s_rem;
    int64_t wgt[kTopkWaves], weq[kTopkWaves];
};

__global__ void __launch_bounds__(kTopkThreads) est_topk_kernel(EstArgs a) {
    __shared__ TopkLds sm;
    const int BH = a.B * a.Hq;
    const bool is_v = blockIdx.x < BH;
    const int bh = is_v ? blockIdx.x : blockIdx.x - BH;
    const int cap = is_v ? a.k_v : a.k_s;
    const double p = is_v ? a.p_v : a.p_s;
    const uint32_t* sc = reinterpret_cast<const uint32_t*>((is_v ? a.v_score : a.s_score) + int64_t(bh) * a.N);
    int32_t* out = (is_v ? a.v_idx : a.s_idx) + int64_t(bh) * cap;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int N = a.N;
    const int n4 = N / 4;
    const u32x4* sc4 = reinterpret_cast<const u32x4*>(sc);

    uint32_t k = uint32_t(cap);
    uint32_t prefix = 0, krem = 0;
    bool selected = false;
    if (p > 0.0) {
        // ---- total mass and the threshold theta = ceil(p T)
        uint64_t t = 0;
        for (int i = tid; i < n4; i += kTopkThreads) {
            const u32x4 x = sc4[i];
            t += mass_fx(x[0]) + mass_fx(x[1]) + mass_fx(x[2]) + mass_fx(x[3]);
        }
        t = wave_sum_u64(t);
        if (lane == 0) sm.wsum[wv] = t;
        __syncthreads();
        uint64_t total = 0;
        for (int w = 0; w < kTopkWaves; ++w) total += sm.wsum[w];
        uint64_t rem = uint64_t(ceil(p * double(total)));
        uint32_t above = 0;   // count of scores above the current prefix
        if (total > 0) {
            uint32_t mask = 0;
            for (int shift = 24; shift >= 0; shift -= 8) {
                for (int i = tid; i < kTopkWaves * kHistStride; i += kTopkThreads) sm.whist[i] = 0;
                for (int i = tid; i < kTopkWaves * 256; i += kTopkThreads) sm.wmass[i] = 0;
                __syncthreads();
                uint32_t* wh = sm.whist + wv * kHistStride;
                uint64_t* wm = sm.wmass + wv * 256;
                for (int i0 = tid; i0 < n4; i0 += 4 * kTopkThreads) {
                    u32x4 x[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int i = i0 + u * kTopkThreads;
                        x[u] = i < n4 ? sc4[i] : u32x4{0u, 0u, 0u, 0u};
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const bool in = i0 + u * kTopkThreads < n4;
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            hist_add_mass(wh, wm, (x[u][e] >> shift) & 255u, mass_fx(x[u][e]),
                                          in && (x[u][e] & mask) == prefix);
                    }
                }
                __syncthreads();
                for (int bb = tid; bb < 256; bb += kTopkThreads) {
                    uint32_t c = 0;
                    uint64_t m = 0;
                    for (int w = 0; w < kTopkWaves; ++w) {
                        c += sm.whist[w * kHistStride + bb];
                        m += sm.wmass[w * 256 + bb];
                    }
                    sm.hist[bb] = c;
                    sm.hmass[bb] = m;
                }
                __syncthreads();
                if (tid == 0) {
                    // the prefix group holds at least rem (> 0): some bin is taken
                    uint64_t run = 0;
                    uint32_t runc = 0;
                    int bsel = 0;
                    for (int bb = 255; bb >= 0; --bb) {
                        if (run + sm.hmass[bb] >= rem) {
                            bsel = bb;
                            break;
                        }
                        run += sm.hmass[bb];
                        runc += sm.hist[bb];
                    }
                    sm.s_prefix = prefix | (uint32_t(bsel) << shift);
                    sm.s_rem = rem - run;
                    sm.s_above = above + runc;
                    if (shift == 0) {
                        // t = the prefix; every score equal to t adds mass_fx(t)
                        const uint64_t qt = mass_fx(sm.s_prefix);
                        const uint64_t ties = qt ? (sm.s_rem + qt - 1) / qt : uint64_t(sm.hist[bsel]);
                        sm.s_k = uint32_t(min<uint64_t>(uint64_t(above + runc) + min<uint64_t>(ties, sm.hist[bsel]),
                                                        uint64_t(N)));
                    }
                }
                __syncthreads();
                prefix = sm.s_prefix;
                rem = sm.s_rem;
                above = sm.s_above;
                mask |= 255u << shift;
                __syncthreads();
            }
            k = sm.s_k;
        } else {
            k = 1;   // no mass at all: one entry reaches p of it
        }
        if (k <= uint32_t(cap)) {
            krem = k - above;
            selected = total > 0;
        } else {
            k = uint32_t(cap);
        }
    }
    if (!selected) {
        prefix = 0;
        uint32_t mask = 0;
        krem = k;
        for (int shift = 24; shift >= 0; shift -= 8) {
            for (int i = tid; i < kTopkWaves * kHistStride; i += kTopkThreads) sm.whist[i] = 0;
            __syncthreads();
            uint32_t* wh = sm.whist + wv * kHistStride;
            for (int i0 = tid; i0 < n4; i0 += 4 * kTopkThreads) {
                u32x4 x[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int i = i0 + u * kTopkThreads;
                    x[u] = i < n4 ? sc4[i] : u32x4{~0u, ~0u, ~0u, ~0u};
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const bool in = i0 + u * kTopkThreads < n4;
#pragma unroll
                    for (int e = 0; e < 4; ++e) hist_add(wh, (x[u][e] >> shift) & 255u, in && (x[u][e] & mask) == prefix);
                }
            }
            __syncthreads();
            for (int bb = tid; bb < 256; bb += kTopkThreads) {
                uint32_t t = 0;
                for (int w = 0; w < kTopkWaves; ++w) t += sm.whist[w * kHistStride + bb];
                sm.hist[bb] = t;
            }
            __syncthreads();
            if (tid == 0) {
                uint32_t run = 0;
                int bsel = 0;
                for (int bb = 255; bb >= 0; --bb) {
                    if (run + sm.hist[bb] >= krem) {
                        bsel = bb;
                        break;
                    }
                    run += sm.hist[bb];
                }
                sm.s_prefix = prefix | (uint32_t(bsel) << shift);
                sm.s_krem = krem - run;
            }
            __syncthreads();
            prefix = sm.s_prefix;
            krem = sm.s_krem;
            mask |= 255u << shift;
            __syncthreads();
        }
    }
    // prefix = bit pattern of the k-th largest; take all above it and the
    // first krem equal ones, in index order.  Wave wv owns the contiguous
    // slice [wv C, (wv + 1) C) and reads it 64 scores at a time (coalesced);
    // ballots give the counts and ranks, one scan over the waves the offsets.
    const int C = ((N + kTopkWaves * 64 - 1) / (kTopkWaves * 64)) * 64;
    const int lo = wv * C, hi = min(N, lo + C);
    const uint64_t below = (1ull << lane) - 1ull;
    int64_t gt = 0, eq = 0;
    for (int i0 = lo; i0 < hi; i0 += 64) {
        const int i = i0 + lane;
        const uint32_t x = i < hi ? sc[i] : 0u;
        gt += __popcll(__ballot(i < hi && x > prefix));
        eq += __popcll(__ballot(i < hi && x == prefix));
    }
    if (lane == 0) {
        sm.wgt[wv] = gt;
        sm.weq[wv] = eq;
    }
    __syncthreads();
    int64_t off = 0, eq_before = 0;
    for (int w = 0; w < wv; ++w) {
        off += sm.wgt[w] + min<int64_t>(sm.weq[w], max<int64_t>(0, int64_t(krem) - eq_before));
        eq_before += sm.weq[w];
    }
    for (int i0 = lo; i0 < hi; i0 += 64) {
        const int i = i0 + lane;
        const uint32_t x = i < hi ? sc[i] : 0u;
        const bool e = i < hi && x == prefix;
        const uint64_t me = __ballot(e);
        const bool take = (i < hi && x > prefix) || (e && eq_before + __popcll(me & below) < int64_t(krem));
        const uint64_t mt = __ballot(take);
        if (take) out[off + __popcll(mt & below)] = i;
        off += __popcll(mt);
        eq_before += __popcll(me);
    }
    if (p > 0.0) {
        for (int i = int(k) + tid; i < cap; i += kTopkThreads) out[i] = -1;
        if (tid == 0) (is_v ? a.v_cnt : a.s_cnt)[bh] = int32_t(k);
    }
}

template <int D>
hipError_t launch_d(const EstArgs& a, hipStream_t s) {
    const int BH = a.B * a.Hq;
    { TraceScope _t("est_pass1", s); hipLaunchKernelGGL(est_pass1_kernel<D>, dim3(BH * a.nchunk), dim3(kThreads), 0, s, a); }
    { TraceScope _t("est_combine", s); hipLaunchKernelGGL(est_combine_kernel, dim3(BH), dim3(64 * kCombineSplit), 0, s, a); }
    { TraceScope _t("est_pass2", s); hipLaunchKernelGGL(est_pass2_kernel<D>, dim3(BH * a.nchunk), dim3(kThreads), 0, s, a); }
    const int64_t n = int64_t(BH) * a.N;
    { TraceScope _t("est_diag", s); hipLaunchKernelGGL(est_diag_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, a); }
    { TraceScope _t("est_topk", s); hipLaunchKernelGGL(est_topk_kernel, dim3(2 * BH), dim3(kTopkThreads), 0, s, a); }
    return hipGetLastError();
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
    a.diag_part = reinterpret_cast<float*>(base + L.diag_part);
}

hipError_t launch_estimate(const EstArgs& a, hipStream_t s) {
    return a.d == 128 ? launch_d<128>(a, s) : launch_d<64>(a, s);
}

}  // namespace msparse
