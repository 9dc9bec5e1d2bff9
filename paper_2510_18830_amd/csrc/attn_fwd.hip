// Sparse attention forward over the selected 64 x 64 blocks and gathered
// vertical columns (block_bar_sparse_attention_forward, Algorithm 2), and the
// log-sum-exp merge of ring-step partials (merge_out_and_lse, Algorithm 2).
//
// One workgroup of two wavefronts per (batch, query head, 64-row query block);
// wave w owns rows 32w .. 32w+31.  Per 64-key tile:
//   S^T = K Q^T       (A = K rows from LDS, B = the wave's Q rows in VGPRs),
//   online softmax    (each lane owns one query row, the partner lane l^32
//                      holds the other half of its keys),
//   O^T += V^T P^T    (A = V^T from the transposed LDS copy, B = P straight
//                      from the S^T accumulator; this product runs in fp16,
//                      whose 3 extra significand bits keep the rounding of P
//                      well below the output tolerance at the same MFMA rate).
// Block tiles come first, then the column list in chunks of 64 gathered keys.
// Scores use exp2 with scale * log2(e) folded in; lse is stored as a natural log.
#include "common.h"
#include "kernels.h"
#include "trace.h"
#include "tiles.h"

namespace msparse {

namespace {

constexpr int kFwdThreads = 128;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kSlack = 8.f;   // log2 units

template <int D>
struct FwdLds {
    uint16_t k[TileLds<D>::kRowElems];
    uint16_t vt[TileLds<D>::kTElems];
    int32_t kidx[64];
    int32_t lim[64];   // key visible to in-block query row r iff r >= lim
};

// Two waves per SIMD (at most 256 registers per lane): the staging of one
// workgroup overlaps the MFMA work of the other.
template <int D>
__global__ void __launch_bounds__(kFwdThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
attn_fwd_kernel(AttnArgs a) {
    constexpr int KD = D / 16;   // k-steps over head_dim
    constexpr int ND = D / 32;   // 32-wide output column blocks
    __shared__ FwdLds<D> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int h = lane >> 5;      // lane half
    const int l32 = lane & 31;

    const int BH = a.B * a.Hq;
    const int64_t t = blockIdx.x;
    const int bh = int(t % BH);
    const int qb = a.nqb - 1 - int(t / BH);   // heaviest (latest) blocks first
    const int b = bh / a.Hq;
    const int hq = bh % a.Hq;
    const int hk = hq / (a.Hq / a.Hkv);
    const int qrow = 32 * w + l32;            // row inside the query block

    const uint16_t* __restrict__ qp = a.q + (int64_t(bh) * a.Nq + int64_t(qb) * 64 + qrow) * D;
    const uint16_t* __restrict__ kp = a.k + (int64_t(b) * a.Hkv + hk) * int64_t(a.Nk) * D;
    const uint16_t* __restrict__ vp = a.v + (int64_t(b) * a.Hkv + hk) * int64_t(a.Nk) * D;

    u32x4 qreg[KD];
#pragma unroll
    for (int s = 0; s < KD; ++s) qreg[s] = *reinterpret_cast<const u32x4*>(qp + 16 * s + 8 * h);

    f32x16 oacc[ND];
#pragma unroll
    for (int i = 0; i < ND; ++i) oacc[i] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;
    const float c2 = a.scale * kLog2e;

    const int64_t item = int64_t(bh) * a.nqb + qb;
    const int64_t b0 = a.blk_ptr[item], b1 = a.blk_ptr[item + 1];
    const int64_t c0 = a.col_ptr[item], c1 = a.col_ptr[item + 1];
    const int nblk = int(b1 - b0);
    const int ncolt = int((c1 - c0 + 63) / 64);
    const int32_t qg = a.q_blk_global[qb];

    for (int tt = 0; tt < nblk + ncolt; ++tt) {
        // ---- tile metadata: key rows and per-key visibility limit
        bool masked;
        int kb = -1;
        if (tt < nblk) {
            kb = a.blk_idx[b0 + tt];
            masked = a.k_blk_global[kb] == qg;    // diagonal tile: causal inside
            if (masked && tid < 64) sm.lim[tid] = tid;
        } else {
            masked = true;
            const int64_t cbase = c0 + int64_t(tt - nblk) * 64;
            const int cnt = int(min<int64_t>(64, c1 - cbase));
            if (tid < 64) {
                const int j = tid < cnt ? tid : 0;
                const int32_t col = a.col_idx[cbase + j];
                sm.kidx[tid] = col;
                sm.lim[tid] = tid < cnt ? (a.k_blk_global[col >> 6] == qg ? (col & 63) : 0) : 64;
            }
            __syncthreads();
        }
        if (kb >= 0) {
            const ContiguousRows rows{int64_t(kb) * 64};
            stage_rows<D, kFwdThreads>(sm.k, kp, rows, tid);
            stage_transposed_f16<D, kFwdThreads>(sm.vt, vp, rows, 1.0f, tid);
        } else {
            stage_rows<D, kFwdThreads>(sm.k, kp, IndexedRows{sm.kidx}, tid);
            stage_transposed_f16<D, kFwdThreads>(sm.vt, vp, IndexedRows{sm.kidx}, 1.0f, tid);
        }
        __syncthreads();

        // ---- S^T for keys 0-31 (c = 0) and 32-63 (c = 1)
        f32x16 sacc[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            sacc[c] = f32x16{};
            const uint16_t* krow = sm.k + (32 * c + l32) * TileLds<D>::kRowStride + 8 * h;
#pragma unroll
            for (int s = 0; s < KD; ++s) sacc[c] = mfma32(lds_read16(krow + 16 * s), qreg[s], sacc[c]);
        }
        // ---- mask, tile max (raw logits; scale > 0 commutes with max)
        if (masked) {
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = 32 * c + 8 * (r >> 2) + 4 * h + (r & 3);
                    if (qrow < sm.lim[key]) sacc[c][r] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[c][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 32)) * c2;
        // Lazy rescaling: keep the running maximum unless the tile exceeds it
        // by more than kSlack (P then stays below 2^kSlack, well inside fp16),
        // so the O accumulator is rescaled only on the rare tiles that raise
        // the row maximum substantially.
        const bool raise = mx > m_run + kSlack;
        if (__any(raise)) {
            const float m_new = raise ? mx : m_run;
            const float alpha = m_run == -INFINITY ? 0.f : fast_exp2(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int i = 0; i < ND; ++i) oacc[i] *= alpha;
            m_run = m_new;
        }
        const float m_use = m_run == -INFINITY ? 0.f : m_run;
        float rs = 0.f;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = fast_exp2(__builtin_fmaf(sacc[c][r], c2, -m_use));
                sacc[c][r] = p;
                rs += p;
            }
        l_run += rs + __shfl_xor(rs, 32);

        // ---- O^T += V^T P^T
        u32x4 pb[4];
        pb[0] = pack8_f16<0>(sacc[0]);
        pb[1] = pack8_f16<8>(sacc[0]);
        pb[2] = pack8_f16<0>(sacc[1]);
        pb[3] = pack8_f16<8>(sacc[1]);
#pragma unroll
        for (int i = 0; i < ND; ++i) {
            const uint16_t* vrow = sm.vt + (32 * i + l32) * TileLds<D>::kTStride + 8 * h;
#pragma unroll
            for (int g = 0; g < 4; ++g) oacc[i] = mfma32h(lds_read16(vrow + 16 * g), pb[g], oacc[i]);
        }
        __syncthreads();
    }

    // ---- epilogue: normalise, store bf16 out and natural-log lse
    const bool empty = !(l_run > 0.f);
    const float inv = empty ? 0.f : 1.f / l_run;
    const int64_t orow = (int64_t(bh) * a.Nq + int64_t(qb) * 64 + qrow) * D;
#pragma unroll
    for (int i = 0; i < ND; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f32x4 o4;
            o4.x = oacc[i][4 * g + 0] * inv;
            o4.y = oacc[i][4 * g + 1] * inv;
            o4.z = oacc[i][4 * g + 2] * inv;
            o4.w = oacc[i][4 * g + 3] * inv;
            if (a.out) {
                u32x2 pk;
                pk.x = pack_bf16x2(o4.x, o4.y);
                pk.y = pack_bf16x2(o4.z, o4.w);
                *reinterpret_cast<u32x2*>(a.out + orow + 32 * i + 8 * g + 4 * h) = pk;
            }
            if (a.out_f32) *reinterpret_cast<f32x4*>(a.out_f32 + orow + 32 * i + 8 * g + 4 * h) = o4;
        }
    if (h == 0) {
        float* lp = a.lse + int64_t(bh) * a.Nq + int64_t(qb) * 64 + qrow;
        *lp = empty ? -INFINITY : (m_run + fast_log2(l_run)) * kLn2;
    }
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
    const int64_t grid = int64_t(a.B) * a.Hq * a.nqb;
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
