// Sparse attention forward over the selected 64 x 64 blocks and gathered
// vertical columns (block_bar_sparse_attention_forward, Algorithm 2), and the
// log-sum-exp merge of ring-step partials (merge_out_and_lse, Algorithm 2).
//
// One workgroup of four wavefronts per (batch, query head, pair of consecutive
// 64-row query blocks); waves 2j, 2j+1 own block j of the pair, 32 rows each.
// The pair walks the union of its two block lists in ascending key order:
// every key tile is staged once, and each half computes it only when its own
// list selected it (the lists of neighbouring blocks share most of their
// tiles: a run of selected diagonals x..x+r gives the pair r+2 distinct key
// blocks for 2(r+1) block products).  Column tiles follow, per half.
// Per 64-key tile, per wave:
//   S^T = K Q^T       (A = K rows from LDS, B = the wave's Q rows in VGPRs),
//   online softmax    (each lane owns one query row, the partner lane l^32
//                      holds the other half of its keys),
//   O^T += V^T P^T    (A = V^T read transposed from fp16 V rows in LDS,
//                      B = P straight from the S^T accumulator; this product
//                      runs in fp16, whose 3 extra significand bits keep the
//                      rounding of P well below the output tolerance at the
//                      same MFMA rate; the fp16 copy of V, times a power of
//                      two sv from max |V|, is made once per call by a
//                      conversion pass and 1/sv applied at the end).
// Scores use exp2 with scale * log2(e) folded in; lse is stored as a natural log.
#include "common.h"
#include "kernels.h"
#include "trace.h"
#include "tiles.h"

namespace msparse {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kSlack = 8.f;   // log2 units

// Online-softmax state of one wave: 32 query rows, O^T accumulator.
template <int D>
struct FwdRows {
    static constexpr int KD = D / 16;   // k-steps over head_dim
    static constexpr int ND = D / 32;   // 32-wide output column blocks
    u32x4 q[KD];
    f32x16 o[ND];
    float m = -INFINITY, l = 0.f;
};

// One 64-key tile for one wave.  lims (LDS, or NULL for a tile without
// masking): key k is visible to in-block query row r iff r >= lims[k] (the
// causal diagonal uses lims[k] = k).  The masking is a rare uniform branch
// whose limits come from LDS, so nothing of it is hoisted into the loop.
template <int D>
__device__ __forceinline__ void fwd_tile(const uint16_t* kt, const uint16_t* vt, const int32_t* lims, FwdRows<D>& st,
                                         int qrow, int lane, float c2) {
    const int h = lane >> 5, l32 = lane & 31;
    constexpr int KD = FwdRows<D>::KD, ND = FwdRows<D>::ND;
    // ---- S^T for keys 0-31 (c = 0) and 32-63 (c = 1)
    // operands read in groups of two k-steps into two register sets, group
    // g + 1 before group g's MFMAs (scheduling fences keep that order), so the
    // LDS latency overlaps the MFMAs
    f32x16 sacc[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) sacc[c] = f32x16{};
    u32x4 fk[2][2][2];   // [set][k-step of group][c]
    auto read_group = [&](int set, int s0) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int c = 0; c < 2; ++c) fk[set][j][c] = dma_read16<D, kRowPad>(kt, 32 * c + l32, h + 2 * (s0 + j));
    };
    read_group(0, 0);
#pragma unroll
    for (int s0 = 0; s0 < KD; s0 += 2) {
        const int set = (s0 >> 1) & 1;
        if (s0 + 2 < KD) read_group(set ^ 1, s0 + 2);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int c = 0; c < 2; ++c) sacc[c] = mfma32(fk[set][j][c], st.q[s0 + j], sacc[c]);
        __builtin_amdgcn_sched_barrier(0);
    }
    // V^T operands in groups of one d block (4 operands) into two register
    // sets; the first group is read now, so its LDS latency is covered by the
    // softmax terms below
    u32x4 av[2][4];
    auto read_tr = [&](int set, int i) {
#pragma unroll
        for (int g = 0; g < 4; ++g) av[set][g] = dma_read_tr<D, kTrPad>(vt, 16 * g, 32 * i, lane);
    };
    read_tr(0, 0);
    __builtin_amdgcn_sched_barrier(0);
    // ---- mask, tile max (raw logits; scale > 0 commutes with max)
    if (lims) {
        keep_branch();
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int k0 = 32 * c + 8 * q4 + 4 * h;
                const i32x4 l4 = *reinterpret_cast<const i32x4*>(lims + k0);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (qrow < l4[e]) sacc[c][4 * q4 + e] = -INFINITY;
            }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[c][r]);
    mx = half_swap_max(mx) * c2;
    // Lazy rescaling: keep the running maximum unless the tile exceeds it by
    // more than kSlack (P then stays below 2^kSlack, well inside fp16), so the
    // O accumulator is rescaled only on the rare tiles that raise the row
    // maximum substantially.
    const bool raise = mx > st.m + kSlack;
    if (__any(raise)) {
        const float m_new = raise ? mx : st.m;
        const float alpha = st.m == -INFINITY ? 0.f : fast_exp2(st.m - m_new);
        st.l *= alpha;
#pragma unroll
        for (int i = 0; i < ND; ++i) st.o[i] *= alpha;
        st.m = m_new;
    }
    const float m_use = st.m == -INFINITY ? 0.f : st.m;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[c][r] = fast_exp2(__builtin_fmaf(sacc[c][r], c2, -m_use));
    // ---- O^T += V^T P^T (A = V^T read transposed from the fp16 V rows)
    u32x4 pb[4];
    pb[0] = pack8_f16<0>(sacc[0]);
    pb[1] = pack8_f16<8>(sacc[0]);
    pb[2] = pack8_f16<0>(sacc[1]);
    pb[3] = pack8_f16<8>(sacc[1]);
    // The normaliser sums the fp16 weights the product uses, so O is an exact
    // convex combination of V rows with those weights: its rounding error then
    // shrinks with the weight outside the largest one, and Delta = dO . O of
    // the backward stays consistent with its own probabilities even for
    // nearly one-hot rows (which would otherwise amplify the 2^-12 rounding
    // of P by 1 / (1 - max P)).
    st.l += row_sum_f16(pb);
#pragma unroll
    for (int i = 0; i < ND; ++i) {
        const int set = i & 1;
        if (i + 1 < ND) read_tr(set ^ 1, i + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int g = 0; g < 4; ++g) st.o[i] = mfma32h(av[set][g], pb[g], st.o[i]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

#ifndef MS_FWD_NB
#define MS_FWD_NB 2
#endif
constexpr int kFwdBlocks = MS_FWD_NB;            // query blocks per workgroup
constexpr int kFwdThreads = 128 * kFwdBlocks;    // two waves per block

// Two waves per SIMD at head dim 128 (at most 256 registers per lane), three
// at 64 (at most 168): the staging and barrier waits of one set of waves
// overlap the MFMA work of another.
// Workgroup = kFwdBlocks consecutive query blocks of one head; the blocks
// walk the union of their ascending block lists (each key tile staged once,
// computed by the blocks whose list selected it), then each block's column
// tiles.
template <int D>
__global__ void __launch_bounds__(kFwdThreads) __attribute__((amdgpu_waves_per_eu(2, D == 64 ? 3 : 2)))
attn_fwd_kernel(AttnArgs a) {
    constexpr int KD = FwdRows<D>::KD, ND = FwdRows<D>::ND;
    constexpr int NB = kFwdBlocks, NW = 2 * NB;
    // two pipeline buffers as separate LDS objects (K bf16, V fp16 rows)
    constexpr int KE = DmaTile<D, kRowPad>::kElems, VE = DmaTile<D, kTrPad>::kElems;
    __shared__ uint16_t k0s[KE], v0s[VE], k1s[KE], v1s[VE];
    __shared__ int32_t kidx[64], lims[64], dlims[64];
    if (index_overflowed(a.overflow)) return;   // incomplete lists: outputs are left untouched

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
    const int blk = w >> 1;       // this wave's query block in the group
    const int h = lane >> 5;      // lane half
    const int l32 = lane & 31;

    const int ngroup = (a.nqb + NB - 1) / NB;
    int bh, qgi;
    query_tile_of(blockIdx.x, a.B, a.Hq, a.Hkv, ngroup, bh, qgi);
    const int b = bh / a.Hq;
    const int hq = bh % a.Hq;
    const int hk = hq / (a.Hq / a.Hkv);
    const int qb0 = NB * qgi;
    const int nblk = min(NB, a.nqb - qb0);                    // blocks present in the group
    const bool live = blk < nblk;
    const int qb = qb0 + (live ? blk : 0);                   // an absent block's waves read block 0 and stay idle
    const int qrow = 32 * (w & 1) + l32;                     // row inside the query block
    const int32_t qg = ldc(a.q_blk_global, qb);

    const uint16_t* __restrict__ kp = a.k + (int64_t(b) * a.Hkv + hk) * int64_t(a.Nk) * D;
    const uint16_t* __restrict__ vp = a.v16 + (int64_t(b) * a.Hkv + hk) * int64_t(a.Nk) * D;

    FwdRows<D> st;
    {
        const uint16_t* __restrict__ qptr = a.q + (int64_t(bh) * a.Nq + int64_t(qb) * 64 + qrow) * D;
#pragma unroll
        for (int s = 0; s < KD; ++s) st.q[s] = *reinterpret_cast<const u32x4*>(qptr + 16 * s + 8 * h);
    }
#pragma unroll
    for (int i = 0; i < ND; ++i) st.o[i] = f32x16{};
    const float c2 = a.scale * kLog2e;

    // ---- block tiles: the union of the NB ascending block lists, software
    // pipelined (the loads of the next tile are in flight during this tile)
    const int64_t item0 = int64_t(bh) * a.nqb + qb0;
    // Lists are walked from their last (nearest the diagonal) tile down: the
    // band of block-diagonals that a KV group's heads share comes first, so
    // the group's workgroups read the same K / V tiles at about the same time
    // (L2 reuse), and the running maximum is set early (fewer rescales).
    int64_t p[NB], e[NB];   // p: next entry (descending), e: first entry
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        e[j] = j < nblk ? ldc(a.blk_ptr, item0 + j) : 0;
        p[j] = j < nblk ? ldc(a.blk_ptr, item0 + j + 1) - 1 : -1;
    }
    auto next = [&](int32_t& kb, uint32_t& sel, int32_t& kg) {
        int32_t k[NB];
        kb = -1;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            k[j] = p[j] >= e[j] ? ldc(a.blk_idx, p[j]) : -1;
            kb = max(kb, k[j]);
        }
        if (kb < 0) return false;
        sel = 0;
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (k[j] == kb) {
                sel |= 1u << j;
                --p[j];
            }
        kg = ldc(a.k_blk_global, kb);
        return true;
    };
    if (tid < 64) dlims[tid] = tid;   // causal diagonal: key k visible to rows >= k
    // The walk runs one tile ahead of the loads: the list entries of tile t + 2
    // are read (scalar loads) after tile t's compute, so they arrive during the
    // end-of-tile wait, and no scalar load is outstanding inside a tile (it
    // would make the LDS operand waits drain completely).
    int32_t kb = 0, kg = 0, kbn = 0, kgn = 0;
    uint32_t sel = 0, seln = 0;
    bool have = next(kb, sel, kg);
    if (have) {
        const ContiguousRows rows{int64_t(kb) * 64};
        dma_rows<D, kRowPad, NW>(k0s, kp, rows, w, lane);
        dma_rows<D, kTrPad, NW>(v0s, vp, rows, w, lane);
    }
    bool haven = have && next(kbn, seln, kgn);
    wait_vmem();
    __syncthreads();
    // one tile: compute from (ck, cv) while the next tile lands in (nk, nv)
    auto step = [&](const uint16_t* ck, const uint16_t* cv, uint16_t* nk, uint16_t* nv) {
        if (haven) {
            const ContiguousRows rows{int64_t(kbn) * 64};
            dma_rows<D, kRowPad, NW>(nk, kp, rows, w, lane);
            dma_rows<D, kTrPad, NW>(nv, vp, rows, w, lane);
        }
        if ((sel >> blk) & 1u) fwd_tile<D>(ck, cv, kg == qg ? dlims : nullptr, st, qrow, lane, c2);
        __builtin_amdgcn_sched_barrier(0);
        int32_t kb2 = 0, kg2 = 0;
        uint32_t sel2 = 0;
        const bool more2 = haven && next(kb2, sel2, kg2);
        wait_vmem();
        __syncthreads();
        kb = kbn;
        kg = kgn;
        sel = seln;
        have = haven;
        kbn = kb2;
        kgn = kg2;
        seln = sel2;
        haven = more2;
    };
    while (have) {
        step(k0s, v0s, k1s, v1s);
        if (!have) break;
        step(k1s, v1s, k0s, v0s);
    }

    // ---- column tiles, one block at a time (the lists differ only near the band)
    for (int j = 0; j < nblk; ++j) {
        const int64_t c0 = ldc(a.col_ptr, item0 + j), c1 = ldc(a.col_ptr, item0 + j + 1);
        const int32_t qgj = ldc(a.q_blk_global, qb0 + j);
        for (int64_t cbase = c0; cbase < c1; cbase += 64) {
            const int cnt = int(min<int64_t>(64, c1 - cbase));
            if (tid < 64) {
                const int32_t col = a.col_idx[cbase + (tid < cnt ? tid : 0)];
                kidx[tid] = col;
                lims[tid] = tid < cnt ? (a.k_blk_global[col >> 6] == qgj ? (col & 63) : 0) : 64;
            }
            __syncthreads();
            dma_rows<D, kRowPad, NW>(k0s, kp, IndexedRows{kidx}, w, lane);
            dma_rows<D, kTrPad, NW>(v0s, vp, IndexedRows{kidx}, w, lane);
            wait_vmem();
            __syncthreads();
            if (blk == j) fwd_tile<D>(k0s, v0s, lims, st, qrow, lane, c2);
            __syncthreads();
        }
    }
    if (!live) return;

    // ---- epilogue: normalise (V carried the factor sv), store bf16 out and
    // natural-log lse; with merge_acc, merge into the running (out_f32, lse)
    // instead (the log-sum-exp merge of ring-step partials, same arithmetic as
    // merge_kernel)
    const bool empty = !(st.l > 0.f);
    const float inv = empty ? 0.f : 1.f / (st.l * operand_scale(a.qkvmax + 2));
    const int64_t lrow = int64_t(bh) * a.Nq + int64_t(qb) * 64 + qrow;
    const int64_t orow = lrow * D;
    const float lp = empty ? -INFINITY : (st.m + fast_log2(st.l)) * kLn2;
    float lnew = lp, wa = 0.f, wp = 1.f, ws = 1.f;
    bool zero = false;
    if (a.merge_acc) {
        const float la = a.lse[lrow];
        const float mx = fmaxf(la, lp);
        if (mx == -INFINITY) {
            lnew = -INFINITY;
            zero = true;
        } else {
            wa = expf(la - mx);
            wp = expf(lp - mx);
            ws = wa + wp;
            lnew = mx + logf(ws);
        }
    }
#pragma unroll
    for (int i = 0; i < ND; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f32x4 o4;
            o4.x = st.o[i][4 * g + 0] * inv;
            o4.y = st.o[i][4 * g + 1] * inv;
            o4.z = st.o[i][4 * g + 2] * inv;
            o4.w = st.o[i][4 * g + 3] * inv;
            float* of = a.out_f32 ? a.out_f32 + orow + 32 * i + 8 * g + 4 * h : nullptr;
            if (a.merge_acc) {
                const f32x4 acc = *reinterpret_cast<const f32x4*>(of);
                o4.x = zero ? 0.f : (wa * acc.x + wp * o4.x) / ws;
                o4.y = zero ? 0.f : (wa * acc.y + wp * o4.y) / ws;
                o4.z = zero ? 0.f : (wa * acc.z + wp * o4.z) / ws;
                o4.w = zero ? 0.f : (wa * acc.w + wp * o4.w) / ws;
            }
            if (a.out) {
                u32x2 pk;
                pk.x = pack_bf16x2(o4.x, o4.y);
                pk.y = pack_bf16x2(o4.z, o4.w);
                *reinterpret_cast<u32x2*>(a.out + orow + 32 * i + 8 * g + 4 * h) = pk;
            }
            if (of) *reinterpret_cast<f32x4*>(of) = o4;
        }
    if (h == 0) a.lse[lrow] = lnew;
}

__global__ void fwd_prep_kernel(AttnArgs a) {
    if (threadIdx.x == 0) a.qkvmax[2] = 0u;
}

__global__ void merge_kernel(MergeArgs m) {
    // one thread per (row, 4 consecutive d)
    const int64_t per_row = m.d / 4;
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= m.rows * per_row) return;
    const int64_t row = i / per_row;
    const int64_t col = (i % per_row) * 4;
    const float lp = m.lse_part[row];
    const f32x4 pk = *reinterpret_cast<const f32x4*>(m.o_part + row * m.d + col);
    float po[4] = {pk.x, pk.y, pk.z, pk.w};
    float res[4];
    float lnew;
    if (m.first) {
        lnew = lp;
        for (int j = 0; j < 4; ++j) res[j] = po[j];
    } else {
        const float la = m.lse_acc[row];
        const float mx = fmaxf(la, lp);
        if (mx == -INFINITY) {
            lnew = -INFINITY;
            for (int j = 0; j < 4; ++j) res[j] = 0.f;
        } else {
            const float wa = expf(la - mx), wp = expf(lp - mx);
            const float s = wa + wp;
            lnew = mx + logf(s);
            const float* acc = m.o_acc + row * m.d + col;
            for (int j = 0; j < 4; ++j) res[j] = (wa * acc[j] + wp * po[j]) / s;
        }
    }
    float* acc = m.o_acc + row * m.d + col;
    for (int j = 0; j < 4; ++j) acc[j] = res[j];
    if (m.out) {
        u32x2 o;
        o.x = pack_bf16x2(res[0], res[1]);
        o.y = pack_bf16x2(res[2], res[3]);
        *reinterpret_cast<u32x2*>(m.out + row * m.d + col) = o;
    }
    if (col == 0) m.lse_acc[row] = lnew;
}

}  // namespace

hipError_t launch_attn_fwd(const AttnArgs& a, hipStream_t s) {
    const int64_t grid = int64_t(a.B) * a.Hq * ((a.nqb + kFwdBlocks - 1) / kFwdBlocks);
    if (grid == 0) return hipSuccess;
    // fp16 copy of V times a power of two from max |V|
    hipLaunchKernelGGL(fwd_prep_kernel, dim3(1), dim3(64), 0, s, a);
    const int64_t nkv = int64_t(a.B) * a.Hkv * a.Nk * a.d;
    hipError_t e = launch_absmax(a.v, nkv, a.qkvmax + 2, s);
    if (e == hipSuccess) e = launch_to_f16(a.v, a.v16, nkv, a.qkvmax + 2, kOperandExp, s);
    if (e != hipSuccess) return e;
    if (a.d == 128)
        { TraceScope _t("attn_fwd", s); hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(unsigned(grid)), dim3(kFwdThreads), 0, s, a); }
    else
        { TraceScope _t("attn_fwd", s); hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(unsigned(grid)), dim3(kFwdThreads), 0, s, a); }
    return hipGetLastError();
}

hipError_t launch_merge(const MergeArgs& m, hipStream_t s) {
    const int64_t n = m.rows * (m.d / 4);
    const int threads = 256;
    { TraceScope _t("merge_out_lse", s); hipLaunchKernelGGL(merge_kernel, dim3(unsigned((n + threads - 1) / threads)), dim3(threads), 0, s, m); }
    return hipGetLastError();
}

}  // namespace msparse
