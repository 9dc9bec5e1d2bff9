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
    const int bh = blockIdx.x / a.nchunk;
    const int chunk = blockIdx.x % a.nchunk;
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

__global__ void __launch_bounds__(64) est_combine_kernel(EstArgs a) {
    const int bh = blockIdx.x, r = threadIdx.x;
    float M = -INFINITY;
    for (int c = 0; c < a.nchunk; ++c) M = fmaxf(M, a.part_max[(int64_t(bh) * a.nchunk + c) * kBlock + r]);
    float S = 0.f;
    for (int c = 0; c < a.nchunk; ++c) {
        const int64_t o = (int64_t(bh) * a.nchunk + c) * kBlock + r;
        const float pm = a.part_max[o];
        if (pm != -INFINITY) S += a.part_sum[o] * fast_exp2(pm - M);
    }
    a.row_lse[bh * kBlock + r] = M + fast_log2(S);
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
    const int bh = blockIdx.x / a.nchunk;
    const int chunk = blockIdx.x % a.nchunk;
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
            // delta_local = r - c = tid - 63
            const int dl = tid - 63;
            const int r0 = max(0, dl), r1 = min(63, 63 + dl);
            float s = 0.f;
            for (int r = r0; r <= r1; ++r) s += sm.p[r][r - dl];
            a.diag_part[(int64_t(bh) * nb + j) * 128 + tid] = s;
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

__device__ int64_t block_excl_scan(int64_t v, int64_t* tmp, int64_t* total) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
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
        for (int k = 0; k < kTopkThreads / 64; ++k) {
            const int64_t t = tmp[k];
            tmp[k] = run;
            run += t;
        }
        tmp[16] = run;
    }
    __syncthreads();
    const int64_t r = tmp[wid] + x - v;
    *total = tmp[16];
    __syncthreads();
    return r;
}

__global__ void __launch_bounds__(kTopkThreads) est_topk_kernel(EstArgs a) {
    __shared__ uint32_t hist[256];
    __shared__ int64_t tmp[17];
    __shared__ uint32_t s_prefix, s_krem;
    const int BH = a.B * a.Hq;
    const bool is_v = blockIdx.x < BH;
    const int bh = is_v ? blockIdx.x : blockIdx.x - BH;
    const int k = is_v ? a.k_v : a.k_s;
    const uint32_t* sc = reinterpret_cast<const uint32_t*>((is_v ? a.v_score : a.s_score) + int64_t(bh) * a.N);
    int32_t* out = (is_v ? a.v_idx : a.s_idx) + int64_t(bh) * k;
    const int tid = threadIdx.x;
    const int N = a.N;

    uint32_t prefix = 0, mask = 0, krem = uint32_t(k);
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += kTopkThreads) hist[i] = 0;
        __syncthreads();
        for (int i = tid; i < N; i += kTopkThreads) {
            const uint32_t x = sc[i];
            if ((x & mask) == prefix) atomicAdd(&hist[(x >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (tid == 0) {
            uint32_t run = 0;
            int bsel = 0;
            for (int bb = 255; bb >= 0; --bb) {
                if (run + hist[bb] >= krem) {
                    bsel = bb;
                    break;
                }
                run += hist[bb];
            }
            s_prefix = prefix | (uint32_t(bsel) << shift);
            s_krem = krem - run;
        }
        __syncthreads();
        prefix = s_prefix;
        krem = s_krem;
        mask |= 255u << shift;
        __syncthreads();
    }
    // prefix = bit pattern of the k-th largest; take all above it and the
    // first krem equal ones, in index order
    const int per = (N + kTopkThreads - 1) / kTopkThreads;
    const int i0 = min(N, tid * per), i1 = min(N, i0 + per);
    int64_t gt = 0, eq = 0;
    for (int i = i0; i < i1; ++i) {
        const uint32_t x = sc[i];
        gt += x > prefix;
        eq += x == prefix;
    }
    int64_t tot;
    const int64_t eq_before = block_excl_scan(eq, tmp, &tot);
    const int64_t eq_take = max<int64_t>(0, min<int64_t>(eq, int64_t(krem) - eq_before));
    int64_t pos = block_excl_scan(gt + eq_take, tmp, &tot);
    int64_t taken_eq = 0;
    for (int i = i0; i < i1; ++i) {
        const uint32_t x = sc[i];
        if (x > prefix || (x == prefix && taken_eq < eq_take)) {
            if (x == prefix) ++taken_eq;
            out[pos++] = i;
        }
    }
}

template <int D>
hipError_t launch_d(const EstArgs& a, hipStream_t s) {
    const int BH = a.B * a.Hq;
    { TraceScope _t("est_pass1", s); hipLaunchKernelGGL(est_pass1_kernel<D>, dim3(BH * a.nchunk), dim3(kThreads), 0, s, a); }
    { TraceScope _t("est_combine", s); hipLaunchKernelGGL(est_combine_kernel, dim3(BH), dim3(64), 0, s, a); }
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
