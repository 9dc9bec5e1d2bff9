// Sparse attention backward over the forward's index (Eq. softmax_gradient and
// Eq. attention_backward; the index is a constant).  With z = scale q k^T,
// P = exp(z - lse) on the executed entries and Delta_n = dO_n . O_n:
//   dV = P^T dO,  dZ = P o (dO V^T - Delta),  dQ = scale dZ K,  dK = scale dZ^T Q.
//
// Launches on the caller's stream, all deterministic (no atomics decide a
// value; the only atomic is an order-free max):
//   init/delta  Delta_n = dO_n . O_n (from the fp32 forward output when given)
//               and max |dO| over the tensor
//   rowprep     per call: lse2 = lse log2(e) and t s Delta per row
//   dq          query-major over the forward's block + column lists; per tile
//               S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dZ^T        (3 GEMMs)
//   dkdv        key-major over 64-key blocks: for every query head of the KV
//               group and every query block that selected this key block (the
//               transposed lists), S = Q K^T, dP = dO V^T, dV^T += dO^T P,
//               dK^T += Q^T dZ (4 GEMMs); dK / dV of the block written once
//   colplan     work list for the vertical columns: chunks of 64 entries of
//               one head's vertical list, each cut into items of a few query
//               blocks (one workgroup)
//   dkdv-col    the same tile body for one item: the chunk's gathered columns
//               against each of the item's query blocks that sees them outside
//               its selected block-diagonals; partials go to the item's slot
//   merge       adds the column partials into dK / dV, heads and items in order.
// The second GEMM of each pair takes fp16 operands (P or dZ, and Q^T, K^T or
// dO^T converted while staging): 3 more significand bits than bf16 at the same
// MFMA rate.  Two powers of two keep the fp16 operands in range whatever the
// scales of dO and V: dO is multiplied by s (max |s dO| in [8, 16)), and dZ
// by t with t d max|V| in [2^9, 2^10) (dz_scale), so that |t s dZ| < 2^15.
// Results are divided by s (dV) or s t (dQ, dK), so inputs scaled by powers
// of two give exactly the rescaled results.
#include "common.h"
#include "kernels.h"
#include "trace.h"
#include "tiles.h"

namespace msparse {

namespace {

constexpr int kThreads = 128;
constexpr float kLog2e = 1.4426950408889634f;

// ------------------------------------------------------------------ Delta
// max-word reset: all four, or only those of K and V when the Q-side data is reused
__global__ void bwd_init_kernel(AttnArgs a) {
    const int i = threadIdx.x;
    if (i < 4 && (!a.reuse_qrows || i >= 2)) (i == 0 ? a.dmax : a.qkvmax + i - 1)[0] = 0u;
}

constexpr int kDeltaBlocks = 2048;

// Delta = dO . O per row and max |dO|.  16 lanes per row, PER = d / 16
// consecutive elements per lane read with one 16- or 8-byte load of dO and
// one or two 16-byte loads of O; a workgroup takes 8 groups of 16 rows per
// grid-stride step and issues all their loads before the arithmetic, so each
// wave has 8 rows' loads in flight.  One max-atomic per workgroup.
template <int PER, bool F32>
__global__ void __launch_bounds__(256) bwd_delta_kernel(AttnArgs a) {
    constexpr int U = 8;
    __shared__ float wmax[4];
    const int64_t rows = int64_t(a.B) * a.Hq * a.Nq;
    const int sub = threadIdx.x & 15;
    float mx = 0.f;
    for (int64_t row0 = int64_t(blockIdx.x) * 16 * U; row0 < rows; row0 += int64_t(gridDim.x) * 16 * U) {
        float gv[U][PER], ov[U][PER];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t row = row0 + 16 * u + (threadIdx.x >> 4);
            const int64_t base = (row < rows ? row : rows - 1) * (16 * PER) + sub * PER;
            if constexpr (PER == 8) {
                const u32x4 g = *reinterpret_cast<const u32x4*>(a.dout + base);
                const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    gv[u][2 * j] = bf16_lo(gw[j]);
                    gv[u][2 * j + 1] = bf16_hi(gw[j]);
                }
            } else {
                const u32x2 g = *reinterpret_cast<const u32x2*>(a.dout + base);
                gv[u][0] = bf16_lo(g.x);
                gv[u][1] = bf16_hi(g.x);
                gv[u][2] = bf16_lo(g.y);
                gv[u][3] = bf16_hi(g.y);
            }
            if constexpr (F32) {
#pragma unroll
                for (int j0 = 0; j0 < PER; j0 += 4) {
                    const f32x4 o = *reinterpret_cast<const f32x4*>(a.o_f32 + base + j0);
                    ov[u][j0] = o.x;
                    ov[u][j0 + 1] = o.y;
                    ov[u][j0 + 2] = o.z;
                    ov[u][j0 + 3] = o.w;
                }
            } else if constexpr (PER == 8) {
                const u32x4 o = *reinterpret_cast<const u32x4*>(a.o + base);
                const uint32_t ow[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    ov[u][2 * j] = bf16_lo(ow[j]);
                    ov[u][2 * j + 1] = bf16_hi(ow[j]);
                }
            } else {
                const u32x2 o = *reinterpret_cast<const u32x2*>(a.o + base);
                ov[u][0] = bf16_lo(o.x);
                ov[u][1] = bf16_hi(o.x);
                ov[u][2] = bf16_lo(o.y);
                ov[u][3] = bf16_hi(o.y);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t row = row0 + 16 * u + (threadIdx.x >> 4);
            float acc = 0.f;
#pragma unroll
            for (int j = 0; j < PER; ++j) {
                acc += ov[u][j] * gv[u][j];
                if (row < rows) mx = fmaxf(mx, fabsf(gv[u][j]));
            }
#pragma unroll
            for (int off = 8; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
            if (row < rows && sub == 0) a.draw[row] = acc;
        }
    }
    mx = wave_max(mx);
    if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
        const float m = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
        atomicMax(a.dmax, __float_as_uint(m));   // m >= 0: bit patterns order like values
    }
}

__device__ __forceinline__ float dout_scale(const uint32_t* dmax) { return pow2_scale(dmax); }

// Per-row values the tiles read, made on every call (the dZ scale t depends
// on this call's V): lse2 = lse log2(e) (+inf for a row without keys, so its
// P is 0) and t s Delta.
__global__ void __launch_bounds__(256) bwd_rowprep_kernel(AttnArgs a) {
    const int64_t rows = int64_t(a.B) * a.Hq * a.Nq;
    const float ts = dout_scale(a.dmax) * dz_scale(a.qkvmax + 2, a.d);
    for (int64_t n = int64_t(blockIdx.x) * 256 + threadIdx.x; n < rows; n += int64_t(gridDim.x) * 256) {
        const float l = a.lse[n];
        a.lse2[n] = l == -INFINITY ? INFINITY : l * kLog2e;
        a.delta[n] = ts * a.draw[n];
    }
}

// ------------------------------------------------------------------ dQ (query-major)
// One workgroup of four waves per pair of consecutive query blocks (as in the
// forward): the pair walks the union of its block lists with the next key
// tile in flight (direct global->LDS loads, double buffer), then the column
// tiles of each block.  Everything runs on the scaled fp16 copies (sq Q,
// sk K, sv V, s dO; powers of two, folded back exactly).  Per tile and wave:
// S^T = K Q^T, dP^T = V dO^T (K, V rows from LDS, Q and dO rows in VGPRs),
// dQ^T += K^T dZ^T (K^T read transposed from the same K tile).
constexpr int kDqThreads = 256;
#ifndef MS_KV_AHEAD
#define MS_KV_AHEAD 1   // dK/dV operand groups read this many groups ahead
#endif

template <int D>
struct DqRows {
    static constexpr int KD = D / 16, ND = D / 32;
    u32x4 q[KD], g[KD];
    f32x16 acc[ND];
    float lse2, dlt;
};

// lims (LDS, or NULL for a tile without masking): key k visible to in-block
// query row r iff r >= lims[k]; a rare uniform branch (see fwd_tile).
// c2 = scale log2(e) / (sq sk); isv = t / sv (turns the dP^T accumulator into t s dP^T)
template <int D>
__device__ __forceinline__ void dq_tile(const uint16_t* kt, const uint16_t* vt, const int32_t* lims, DqRows<D>& st,
                                        int qrow, int lane, float c2, float isv) {
    constexpr int KD = DqRows<D>::KD, ND = DqRows<D>::ND;
    const int h = lane >> 5, l32 = lane & 31;
    // Two waves per SIMD (the other wave's MFMAs overlap this wave's softmax
    // terms), so the key halves c run one after the other and only one half's
    // S^T / dP^T accumulators are live: S^T, dP^T of keys 32 c .. 32 c + 31,
    // the dZ terms, then that half's dQ k-steps.  Each S / dP k-step's operands
    // are read one step ahead into a second register set.
    u32x4 fk[2], fv[2], ak[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        f32x16 sa = f32x16{}, pa = f32x16{};
        auto read_sd = [&](int set, int s) {
            fk[set] = dma_read16<D, kDualPad>(kt, 32 * c + l32, h + 2 * s);
            fv[set] = dma_read16<D, kDualPad>(vt, 32 * c + l32, h + 2 * s);
        };
        auto read_tr = [&](int i) {
#pragma unroll
            for (int j = 0; j < 2; ++j) ak[j] = dma_read_tr<D, kDualPad>(kt, 16 * (2 * c + j), 32 * i, lane);
        };
        read_sd(0, 0);
#pragma unroll
        for (int k = 0; k < KD; ++k) {
            const int set = k & 1;
            if (k + 1 < KD) read_sd(set ^ 1, k + 1);
            else read_tr(0);
            __builtin_amdgcn_sched_barrier(0);
            sa = mfma32h(fk[set], st.q[k], sa);
            pa = mfma32h(fv[set], st.g[k], pa);
            __builtin_amdgcn_sched_barrier(0);
        }
        // t s dZ^T = P o (t s dP^T - t s Delta), P = exp2(c2 z - lse2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float p = fast_exp2(__builtin_fmaf(sa[r], c2, -st.lse2));
            sa[r] = p * __builtin_fmaf(pa[r], isv, -st.dlt);
        }
        if (lims) {
            keep_branch();
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const i32x4 l4 = *reinterpret_cast<const i32x4*>(lims + 32 * c + 8 * q4 + 4 * h);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (qrow < l4[e]) sa[4 * q4 + e] = 0.f;
            }
        }
        u32x4 zb[2];
        zb[0] = pack8_f16<0>(sa);
        zb[1] = pack8_f16<8>(sa);
#pragma unroll
        for (int i = 0; i < ND; ++i) {
            if (i > 0) read_tr(i);
#pragma unroll
            for (int j = 0; j < 2; ++j) st.acc[i] = mfma32h(ak[j], zb[j], st.acc[i]);
        }
    }

}

// Two waves per SIMD at head dim 128, three at 64 (168 registers; the few
// spilled values cost less than the third wave gains: 17.9 -> 16.6 ms on the
// 128K layer's shape at d 64).
template <int D>
__global__ void __launch_bounds__(kDqThreads)
    __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2, D == 64 ? 3 : 2))) bwd_dq_kernel(AttnArgs a) {
    constexpr int KD = DqRows<D>::KD, ND = DqRows<D>::ND;
    constexpr int TE = DmaTile<D, kDualPad>::kElems;
    __shared__ uint16_t k0s[TE], v0s[TE], k1s[TE], v1s[TE];
    __shared__ int32_t kidx[64], lims[64], dlims[64];
    if (index_overflowed(a.overflow)) return;   // incomplete lists: outputs are left untouched
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), half = w >> 1;
    const int npair = (a.nqb + 1) >> 1;
    if (tid < 64) dlims[tid] = tid;   // causal diagonal: key k visible to rows >= k
    int bh, qp;
    query_tile_of(blockIdx.x, a.B, a.Hq, a.Hkv, npair, bh, qp);
    const int b = bh / a.Hq, hq = bh % a.Hq, hk = hq / (a.Hq / a.Hkv);
    const int qb0 = 2 * qp;
    const bool has1 = qb0 + 1 < a.nqb;
    const int qb = qb0 + (has1 ? half : 0);
    const bool live = half == 0 || has1;
    const int qrow = 32 * (w & 1) + l32;
    const int64_t grow = int64_t(bh) * a.Nq + int64_t(qb) * 64 + qrow;
    const int32_t qg = ldc(a.q_blk_global, qb);
    const float pt = dz_scale(a.qkvmax + 2, D);   // the tiles give t s dZ

    const int64_t kvoff = (int64_t(b) * a.Hkv + hk) * int64_t(a.Nk) * D;
    const uint16_t* __restrict__ kp = a.k16 + kvoff;
    const uint16_t* __restrict__ vp = a.v16 + kvoff;
    DqRows<D> st;
#pragma unroll
    for (int s = 0; s < KD; ++s) {
        st.q[s] = *reinterpret_cast<const u32x4*>(a.q16 + grow * D + 16 * s + 8 * h);
        st.g[s] = *reinterpret_cast<const u32x4*>(a.g16 + grow * D + 16 * s + 8 * h);
    }
    const float sq = operand_scale(a.qkvmax), sk = operand_scale(a.qkvmax + 1);
    const float isv = dz_scale(a.qkvmax + 2, D) / operand_scale(a.qkvmax + 2);   // t / sv
    const float c2 = a.scale * kLog2e / (sq * sk);
    st.lse2 = a.lse2[grow];
    const float sc = dout_scale(a.dmax);
    st.dlt = a.delta[grow];
#pragma unroll
    for (int i = 0; i < ND; ++i) st.acc[i] = f32x16{};

    // ---- block tiles: union of the two ascending block lists, pipelined
    const int64_t item0 = int64_t(bh) * a.nqb + qb0;
    const int64_t e00 = ldc(a.blk_ptr, item0), e01 = ldc(a.blk_ptr, item0 + 1);
    const int64_t e11 = has1 ? ldc(a.blk_ptr, item0 + 2) : e01;
    // walked from the diagonal down (as in the forward: the group's shared
    // band first)
    int64_t p0 = e01 - 1, p1 = e11 - 1;
    auto next = [&](int32_t& kb, bool& in0, bool& in1, bool& diag) {
        if (p0 < e00 && p1 < e01) return false;
        const int32_t k0 = p0 >= e00 ? ldc(a.blk_idx, p0) : -1;
        const int32_t k1 = p1 >= e01 ? ldc(a.blk_idx, p1) : -1;
        kb = max(k0, k1);
        in0 = k0 == kb;
        in1 = k1 == kb;
        p0 -= in0;
        p1 -= in1;
        diag = ldc(a.k_blk_global, kb) == qg;
        return true;
    };
    auto load = [&](uint16_t* kt, uint16_t* vt, auto rows) {
        dma_rows<D, kDualPad, 4>(kt, kp, rows, w, lane);
        dma_rows<D, kDualPad, 4>(vt, vp, rows, w, lane);
    };
    // the walk runs one tile ahead of the loads (as in the forward): no scalar
    // load is outstanding inside a tile
    int32_t kb = 0, kbn = 0;
    bool in0 = false, in1 = false, diag = false, in0n = false, in1n = false, diagn = false;
    bool have = next(kb, in0, in1, diag);
    if (have) load(k0s, v0s, ContiguousRows{int64_t(kb) * 64});
    bool haven = have && next(kbn, in0n, in1n, diagn);
    wait_vmem();
    __syncthreads();
    auto step = [&](const uint16_t* ck, const uint16_t* cv, uint16_t* nk, uint16_t* nv) {
        if (haven) load(nk, nv, ContiguousRows{int64_t(kbn) * 64});
        if (half == 0 ? in0 : in1) dq_tile<D>(ck, cv, diag ? dlims : nullptr, st, qrow, lane, c2, isv);
        __builtin_amdgcn_sched_barrier(0);
        int32_t kb2 = 0;
        bool in02 = false, in12 = false, diag2 = false;
        const bool more2 = haven && next(kb2, in02, in12, diag2);
        wait_vmem();
        __syncthreads();
        kb = kbn;
        in0 = in0n;
        in1 = in1n;
        diag = diagn;
        have = haven;
        kbn = kb2;
        in0n = in02;
        in1n = in12;
        diagn = diag2;
        haven = more2;
    };
    while (have) {
        step(k0s, v0s, k1s, v1s);
        if (!have) break;
        step(k1s, v1s, k0s, v0s);
    }

    // ---- column tiles, one half at a time
    for (int j = 0; j < 1 + int(has1); ++j) {
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
            load(k0s, v0s, IndexedRows{kidx});
            wait_vmem();
            __syncthreads();
            if (half == j) dq_tile<D>(k0s, v0s, lims, st, qrow, lane, c2, isv);
            __syncthreads();
        }
    }
    if (!live) return;
    float* dq = a.dq + grow * D;
    const float fin = a.scale / (sc * pt * sk);
#pragma unroll
    for (int i = 0; i < ND; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f32x4 val;
            val.x = st.acc[i][4 * g + 0] * fin;
            val.y = st.acc[i][4 * g + 1] * fin;
            val.z = st.acc[i][4 * g + 2] * fin;
            val.w = st.acc[i][4 * g + 3] * fin;
            f32x4* dst = reinterpret_cast<f32x4*>(dq + 32 * i + 8 * g + 4 * h);
            if (a.dq_accumulate) val += *dst;
            *dst = val;
        }
}

// ------------------------------------------------------------------ dK / dV (key-major)
// A query tile as the key-major passes stage it (DMA tiles): the scaled fp16
// Q and dO rows, read row-wise for the first GEMMs and transposed for the
// second, and the rows' lse2 and s Delta (64 floats each).
template <int D>
struct KvTile {
    static constexpr int kPart = DmaTile<D, kDualPad>::kElems;
    static constexpr int kElems = 2 * kPart + 256;   // + 128 floats
    // element offsets of the parts
    static constexpr int kQ16 = 0, kG16 = kPart, kRw = 2 * kPart;
};

// Issue the loads of query tile (bh, qb) into tile `t` (NW waves).
template <int D, int NW>
__device__ __forceinline__ void kv_load_query_tile(uint16_t* t, const AttnArgs& a, int bh, int qb, int wave,
                                                   int lane) {
    using T = KvTile<D>;
    const int64_t row0 = int64_t(bh) * a.Nq + int64_t(qb) * 64;
    const ContiguousRows rows{row0};
    dma_rows<D, kDualPad, NW>(t + T::kQ16, a.q16, rows, wave, lane);
    dma_rows<D, kDualPad, NW>(t + T::kG16, a.g16, rows, wave, lane);
    if (wave == 0 && lane < 32) {   // lse2 -> floats 0..63, s Delta -> floats 64..127
        const float* src = lane < 16 ? a.lse2 + row0 + 4 * lane : a.delta + row0 + 4 * (lane - 16);
        dma16(src, lds_addr(t + T::kRw));
    }
}

// One 64-row query tile against this wave's 32 keys, for the column pass
// (one wave per SIMD; `key` = this lane's key inside the 64-key chunk; kreg,
// vreg its scaled fp16 K and V rows).  c2 =
// scale log2(e) / (sq sk); isv = t / sv turns the dP accumulator into t s dP.  lims (LDS, or NULL for a tile without masking):
// the key is visible to in-block query row r iff r >= lims[key] (64: not
// visible); a rare uniform branch whose limit comes from LDS, so nothing of
// it is hoisted into the loop.
// SPLIT: P and t s dZ enter the dV / dK products as two fp16 parts each
// (x = hi + lo, hi = fp16(x), lo = fp16(x - hi); about 22 significand bits):
// the column pass carries most of a vertical key's rows (hundreds of
// thousands at long lengths), where one fp16 rounding of every term would add
// up to errors near the parity bar; it costs two more MFMAs per group there.
template <int D, bool SPLIT = false>
__device__ __forceinline__ void kv_tile(const uint16_t* t, const u32x4* kreg, const u32x4* vreg, const int32_t* lims,
                                        int key, float c2, float isv, int lane, f32x16* dv, f32x16* dk) {
    using T = KvTile<D>;
    constexpr int KD = D / 16, ND = D / 32;
    const int h = lane >> 5, l32 = lane & 31;
    const float* lse2 = reinterpret_cast<const float*>(t + T::kRw);
    const float* dlt = lse2 + 64;
    f32x16 sacc[2], pacc[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        sacc[rb] = f32x16{};
        pacc[rb] = f32x16{};
    }
    // Schedule (one wave per SIMD, so MFMA and VALU overlap only inside the
    // wave's own instruction stream):
    //   A  S, dP of row half 0
    //   B  S, dP of row half 1, interleaved with half 0's softmax terms
    //   C  dV, dK of half 0, interleaved with half 1's softmax terms
    //   D  dV, dK of half 1
    // MFMA operands are read from LDS one group ahead into two register sets;
    // scheduling fences separate the groups (the default schedule waits for
    // every read right before its MFMA and runs the phases back to back).
    // Rows of acc element r: 32 rb + 8 (r/4) + 4 h + r%4; column = this lane's key.
    // Operand groups are read kAhead groups before their MFMAs, into rings of
    // kAhead + 1 register sets (S / dP operands and transposed dV / dK
    // operands); the first transposed groups are read during the last S / dP
    // groups.
    constexpr int kAhead = MS_KV_AHEAD < KD / 2 ? MS_KV_AHEAD : KD / 2, kSets = kAhead + 1;
    u32x4 fq[kSets][2], fg[kSets][2];   // [set][k-step of group]
    auto read_sd = [&](int n) {          // S / dP group n: half n / NG, k-steps 2 (n % NG) + {0, 1}
        const int set = n % kSets, rb = n / (KD / 2), s0 = 2 * (n % (KD / 2));
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            fq[set][j] = dma_read16<D, kDualPad>(t + T::kQ16, 32 * rb + l32, h + 2 * (s0 + j));
            fg[set][j] = dma_read16<D, kDualPad>(t + T::kG16, 32 * rb + l32, h + 2 * (s0 + j));
        }
    };
    auto mfma_sd = [&](int n) {
        const int set = n % kSets, rb = n / (KD / 2), s0 = 2 * (n % (KD / 2));
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            sacc[rb] = mfma32h(fq[set][j], kreg[s0 + j], sacc[rb]);
            pacc[rb] = mfma32h(fg[set][j], vreg[s0 + j], pacc[rb]);
        }
    };
    // P and s dZ of half rb as the fp16 B operands of dV / dK (pb, zb: element
    // r of the accumulator goes to half r % 2 of word (r % 8) / 2 of operand
    // r / 8), written straight from the softmax terms, so the accumulators are
    // never written back
    u32x4 pb[2][2], zb[2][2];   // [rb][j]
    u32x4 pl[SPLIT ? 2 : 1][2], zl[SPLIT ? 2 : 1][2];   // low parts (SPLIT)
    // softmax terms of rows 32 rb + 8 q4 + 4 h + 0..3
    auto soft = [&](int rb, int q4) {
        const int row0 = 32 * rb + 8 * q4 + 4 * h;
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse2 + row0);
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(dlt + row0);
        float pv[4], zv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = 4 * q4 + e;
            pv[e] = fast_exp2(__builtin_fmaf(sacc[rb][r], c2, -l4[e]));
            zv[e] = pv[e] * __builtin_fmaf(pacc[rb][r], isv, -d4[e]);
        }
        const int j = q4 >> 1, w0 = 2 * (q4 & 1);
        pb[rb][j][w0] = pack_f16x2(pv[0], pv[1]);
        pb[rb][j][w0 + 1] = pack_f16x2(pv[2], pv[3]);
        zb[rb][j][w0] = pack_f16x2(zv[0], zv[1]);
        zb[rb][j][w0 + 1] = pack_f16x2(zv[2], zv[3]);
        if constexpr (SPLIT) {
            float plo[4], zlo[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                plo[e] = pv[e] - float(_Float16(pv[e]));
                zlo[e] = zv[e] - float(_Float16(zv[e]));
            }
            const int r2 = SPLIT ? rb : 0;
            pl[r2][j][w0] = pack_f16x2(plo[0], plo[1]);
            pl[r2][j][w0 + 1] = pack_f16x2(plo[2], plo[3]);
            zl[r2][j][w0] = pack_f16x2(zlo[0], zlo[1]);
            zl[r2][j][w0 + 1] = pack_f16x2(zlo[2], zlo[3]);
        }
    };
    // masked entries (rare diagonal tiles): clear their fp16 halves
    auto mask = [&](int rb) {
        if (lims) {
            keep_branch();
            const int lim = lims[key] - 4 * h - 32 * rb;   // row 32 rb + 8 (r/4) + 4 h + r%4 < lims[key]
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (8 * (r >> 2) + (r & 3) < lim) {
                    const uint32_t keep = (r & 1) ? 0x0000FFFFu : 0xFFFF0000u;
                    pb[rb][r >> 3][(r & 7) >> 1] &= keep;
                    zb[rb][r >> 3][(r & 7) >> 1] &= keep;
                    if constexpr (SPLIT) {
                        pl[SPLIT ? rb : 0][r >> 3][(r & 7) >> 1] &= keep;
                        zl[SPLIT ? rb : 0][r >> 3][(r & 7) >> 1] &= keep;
                    }
                }
        }
    };
    // transposed A operands of dV (s dO)^T and dK Q^T for one 32-wide d block
    u32x4 av[kSets][2], ak[kSets][2];   // [set][j]
    auto read_tr = [&](int m) {            // dV / dK group m: half m / ND, d block m % ND
        const int set = m % kSets, rb = m / ND, i = m % ND;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            av[set][j] = dma_read_tr<D, kDualPad>(t + T::kG16, 16 * (2 * rb + j), 32 * i, lane);
            ak[set][j] = dma_read_tr<D, kDualPad>(t + T::kQ16, 16 * (2 * rb + j), 32 * i, lane);
        }
    };
    auto mfma_kv = [&](int m) {
        const int set = m % kSets, rb = m / ND, i = m % ND;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            dv[i] = mfma32h(av[set][j], pb[rb][j], dv[i]);
            dk[i] = mfma32h(ak[set][j], zb[rb][j], dk[i]);
            if constexpr (SPLIT) {
                dv[i] = mfma32h(av[set][j], pl[SPLIT ? rb : 0][j], dv[i]);
                dk[i] = mfma32h(ak[set][j], zl[SPLIT ? rb : 0][j], dk[i]);
            }
        }
    };
    static_assert(KD == 2 * ND, "four S/dP groups and four dV/dK groups per half");
    constexpr int NG = KD / 2;   // groups per half (4 for d = 128)
    constexpr int NSD = 2 * NG, NTR = 2 * ND;
    static_assert(kAhead >= 1 && kAhead <= NG && kAhead <= ND, "read distance");
    // reads issued at S / dP group n: group n + kAhead, or the first transposed groups
    auto ahead_sd = [&](int n) {
        if (n + kAhead < NSD) read_sd(n + kAhead);
        else read_tr(n + kAhead - NSD);
    };
#pragma unroll
    for (int n = 0; n < kAhead; ++n) read_sd(n);
    // ---- A
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        ahead_sd(g);
        __builtin_amdgcn_sched_barrier(0);
        mfma_sd(g);
        __builtin_amdgcn_sched_barrier(0);
    }
    // ---- B
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        ahead_sd(NG + g);
        __builtin_amdgcn_sched_barrier(0);
        mfma_sd(NG + g);
        if (g < 4) soft(0, g);
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int q4 = NG; q4 < 4; ++q4) soft(0, q4);   // d = 64: two groups per half
    mask(0);
    // ---- C
#pragma unroll
    for (int i = 0; i < ND; ++i) {
        if (i + kAhead < NTR) read_tr(i + kAhead);
        __builtin_amdgcn_sched_barrier(0);
        mfma_kv(i);
        if (i < 4) soft(1, i);
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int q4 = ND; q4 < 4; ++q4) soft(1, q4);
    mask(1);
    // ---- D
#pragma unroll
    for (int i = 0; i < ND; ++i) {
        if (ND + i + kAhead < NTR) read_tr(ND + i + kAhead);
        __builtin_amdgcn_sched_barrier(0);
        mfma_kv(ND + i);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// ------------------------------------------------------------------ dK / dV, two waves per SIMD
// Key-major pass: one workgroup of eight waves per (b, KV head, pair of
// consecutive 64-key blocks).  For every query head of the KV group the pair
// walks the union of its two transposed lists (query blocks that selected the
// key block), the next query tile in flight (direct global->LDS loads, double
// buffer) during the current one.  Wave (blk, kh, rh) holds the 32 keys
// 32 kh .. 32 kh + 31 of key block blk of the pair (K in registers) and takes
// rows 32 rh .. 32 rh + 31 of every query tile, so each wave reads only its
// own query rows (row-wise and transposed) and V sits in LDS (staged once per
// workgroup): that leaves room for two waves per SIMD, one wave's MFMAs
// covering the other's softmax terms and LDS latency.  The two row halves'
// partial dK / dV are added once at the end (through LDS, in a fixed order).
constexpr int kKvRowsThreads = 512;

// Rows 32 rh .. 32 rh + 31 of query tile t against this wave's 32 keys, in
// three phases: rows_s_dp (MFMA) forms S = Q K^T (K in registers) and
// dP = dO V^T (V rows of the key block from LDS); rows_terms (VALU) turns them
// into P and t s dZ as fp16 B operands; rows_dv_dk (MFMA) adds
// dV^T += (s dO)^T P and dK^T += Q^T dZ over those rows.
template <int D>
__device__ __forceinline__ void rows_s_dp(const uint16_t* t, const u32x4* kreg, const uint16_t* vt, int key, int rh,
                                          int lane, f32x16& sacc, f32x16& pacc) {
    using T = KvTile<D>;
    constexpr int KD = D / 16;
    const int h = lane >> 5, l32 = lane & 31;
    sacc = f32x16{};
    pacc = f32x16{};
    u32x4 fq[2], fg[2], fv[2];
    auto rd = [&](int set, int s) {
        fq[set] = dma_read16<D, kDualPad>(t + T::kQ16, 32 * rh + l32, h + 2 * s);
        fg[set] = dma_read16<D, kDualPad>(t + T::kG16, 32 * rh + l32, h + 2 * s);
        fv[set] = dma_read16<D, kRowPad>(vt, key, h + 2 * s);
    };
    rd(0, 0);
#pragma unroll
    for (int s = 0; s < KD; ++s) {
        const int set = s & 1;
        if (s + 1 < KD) rd(set ^ 1, s + 1);
        __builtin_amdgcn_sched_barrier(0);
        sacc = mfma32h(fq[set], kreg[s], sacc);
        pacc = mfma32h(fg[set], fv[set], pacc);
        __builtin_amdgcn_sched_barrier(0);
    }
}

template <int D>
__device__ __forceinline__ void rows_terms(const uint16_t* t, const int32_t* lims, int key, int rh, float c2,
                                           float isv, int lane, const f32x16& sacc, const f32x16& pacc, u32x4* pb,
                                           u32x4* zb) {
    using T = KvTile<D>;
    const int h = lane >> 5;
    const float* lse2 = reinterpret_cast<const float*>(t + T::kRw);
    const float* dlt = lse2 + 64;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
        const int row0 = 32 * rh + 8 * q4 + 4 * h;
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse2 + row0);
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(dlt + row0);
        float pv[4], zv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = 4 * q4 + e;
            pv[e] = fast_exp2(__builtin_fmaf(sacc[r], c2, -l4[e]));
            zv[e] = pv[e] * __builtin_fmaf(pacc[r], isv, -d4[e]);
        }
        const int j = q4 >> 1, w0 = 2 * (q4 & 1);
        pb[j][w0] = pack_f16x2(pv[0], pv[1]);
        pb[j][w0 + 1] = pack_f16x2(pv[2], pv[3]);
        zb[j][w0] = pack_f16x2(zv[0], zv[1]);
        zb[j][w0 + 1] = pack_f16x2(zv[2], zv[3]);
    }
    if (lims) {   // rare diagonal tiles: row 32 rh + 8 (r/4) + 4 h + r%4 < lims[key] is masked
        keep_branch();
        const int lim = lims[key] - 4 * h - 32 * rh;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            if (8 * (r >> 2) + (r & 3) < lim) {
                const uint32_t keep = (r & 1) ? 0x0000FFFFu : 0xFFFF0000u;
                pb[r >> 3][(r & 7) >> 1] &= keep;
                zb[r >> 3][(r & 7) >> 1] &= keep;
            }
    }
}

template <int D>
__device__ __forceinline__ void rows_dv_dk(const uint16_t* t, int rh, int lane, const u32x4* pb, const u32x4* zb,
                                           f32x16* dv, f32x16* dk) {
    using T = KvTile<D>;
    constexpr int ND = D / 32;
    u32x4 av[2][2], ak[2][2];   // [set][j]: transposed dO^T / Q^T of one 32-wide d block
    auto rt = [&](int set, int i) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            av[set][j] = dma_read_tr<D, kDualPad>(t + T::kG16, 32 * rh + 16 * j, 32 * i, lane);
            ak[set][j] = dma_read_tr<D, kDualPad>(t + T::kQ16, 32 * rh + 16 * j, 32 * i, lane);
        }
    };
    rt(0, 0);
#pragma unroll
    for (int i = 0; i < ND; ++i) {
        const int set = i & 1;
        if (i + 1 < ND) rt(set ^ 1, i + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            dv[i] = mfma32h(av[set][j], pb[j], dv[i]);
            dk[i] = mfma32h(ak[set][j], zb[j], dk[i]);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

template <int D>
__device__ __forceinline__ void kv_tile_rows(const uint16_t* t, const u32x4* kreg, const uint16_t* vt,
                                             const int32_t* lims, int key, int rh, float c2, float isv, int lane,
                                             f32x16* dv, f32x16* dk) {
    f32x16 sacc, pacc;
    rows_s_dp<D>(t, kreg, vt, key, rh, lane, sacc, pacc);
    u32x4 pb[2], zb[2];
    rows_terms<D>(t, lims, key, rh, c2, isv, lane, sacc, pacc, pb, zb);
    rows_dv_dk<D>(t, rh, lane, pb, zb, dv, dk);
}

template <int D>
__global__ void __launch_bounds__(kKvRowsThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
bwd_dkdv_rows_kernel(AttnArgs a) {
    constexpr int KD = D / 16, ND = D / 32;
    constexpr int TE = KvTile<D>::kElems, VE = DmaTile<D, kRowPad>::kElems;
    // two query-tile buffers (reused at the end for the row halves' reduction)
    __shared__ __attribute__((aligned(16))) uint16_t tb[2 * TE];
    __shared__ __attribute__((aligned(16))) uint16_t vsm[2 * VE];
    __shared__ int32_t dlims[64];
    if (index_overflowed(a.overflow)) return;   // incomplete lists: outputs are left untouched
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = w >> 2, kh = (w >> 1) & 1, rh = w & 1;
    if (tid < 64) dlims[tid] = tid;   // causal diagonal: key k visible to rows >= k
    const int BK = a.B * a.Hkv;
    const int npair = (a.nkb + 1) >> 1;
    const int64_t u = xcd_chunk(blockIdx.x, int64_t(BK) * npair);
    const int bk = int(u / npair);
    const int kp = int(u % npair);
    const int b = bk / a.Hkv, hk = bk % a.Hkv;
    const int G = a.Hq / a.Hkv;
    const int kb0 = 2 * kp;
    const bool has1 = kb0 + 1 < a.nkb;
    const int kb = kb0 + (has1 ? half : 0);
    const bool live = half == 0 || has1;
    const int key = 32 * kh + l32;
    const int64_t krow = int64_t(bk) * a.Nk + int64_t(kb) * 64 + key;
    u32x4 kreg[KD];
#pragma unroll
    for (int s = 0; s < KD; ++s) kreg[s] = *reinterpret_cast<const u32x4*>(a.k16 + krow * D + 16 * s + 8 * h);
    // V rows of the pair's key blocks (a lone block stages it twice)
    dma_rows<D, kRowPad, 8>(vsm, a.v16 + int64_t(bk) * a.Nk * D, ContiguousRows{int64_t(kb0) * 64}, w, lane);
    dma_rows<D, kRowPad, 8>(vsm + VE, a.v16 + int64_t(bk) * a.Nk * D,
                            ContiguousRows{int64_t(has1 ? kb0 + 1 : kb0) * 64}, w, lane);
    const uint16_t* vt = vsm + half * VE;
    f32x16 dv[ND], dk[ND];
#pragma unroll
    for (int i = 0; i < ND; ++i) {
        dv[i] = f32x16{};
        dk[i] = f32x16{};
    }
    const float sq = operand_scale(a.qkvmax), sk = operand_scale(a.qkvmax + 1);
    const float isv = dz_scale(a.qkvmax + 2, D) / operand_scale(a.qkvmax + 2);   // t / sv
    const float c2 = a.scale * kLog2e / (sq * sk);
    const float sc = dout_scale(a.dmax);
    const int32_t kg = ldc(a.k_blk_global, kb);

    // walk: heads of the group in order, per head the union of the pair's two
    // transposed lists
    int g = 0;
    int64_t p0 = 0, e0 = 0, p1 = 0, e1 = 0;
    auto open_head = [&]() {
        const int64_t item = int64_t(b * a.Hq + hk * G + g) * a.nkb + kb0;
        p0 = ldc(a.kblk_ptr, item);
        e0 = ldc(a.kblk_ptr, item + 1);
        p1 = e0;
        e1 = has1 ? ldc(a.kblk_ptr, item + 2) : e0;
    };
    open_head();
    auto next = [&](int& bh, int& qb, bool& in0, bool& in1, bool& diag) {
        while (p0 >= e0 && p1 >= e1) {
            if (++g >= G) return false;
            open_head();
        }
        const int32_t q0 = p0 < e0 ? ldc(a.kblk_idx, p0) : INT32_MAX;
        const int32_t q1 = p1 < e1 ? ldc(a.kblk_idx, p1) : INT32_MAX;
        qb = min(q0, q1);
        in0 = q0 == qb;
        in1 = q1 == qb;
        p0 += in0;
        p1 += in1;
        bh = b * a.Hq + hk * G + g;
        diag = ldc(a.q_blk_global, qb) == kg;
        return true;
    };
    uint16_t* t0s = tb;
    uint16_t* t1s = tb + TE;
    int bh = 0, qb = 0, bhn = 0, qbn = 0;
    bool in0 = false, in1 = false, diag = false, in0n = false, in1n = false, diagn = false;
    bool have = next(bh, qb, in0, in1, diag);
    if (have) kv_load_query_tile<D, 8>(t0s, a, bh, qb, w, lane);
    bool haven = have && next(bhn, qbn, in0n, in1n, diagn);
    wait_vmem();
    __syncthreads();
    auto step = [&](const uint16_t* ct, uint16_t* nt) {
        if (haven) kv_load_query_tile<D, 8>(nt, a, bhn, qbn, w, lane);
        if (half == 0 ? in0 : in1) kv_tile_rows<D>(ct, kreg, vt, diag ? dlims : nullptr, key, rh, c2, isv, lane, dv, dk);
        __builtin_amdgcn_sched_barrier(0);
        int bh2 = 0, qb2 = 0;
        bool in02 = false, in12 = false, diag2 = false;
        const bool more2 = haven && next(bh2, qb2, in02, in12, diag2);
        wait_vmem();
        __syncthreads();
        bh = bhn;
        qb = qbn;
        in0 = in0n;
        in1 = in1n;
        diag = diagn;
        have = haven;
        bhn = bh2;
        qbn = qb2;
        in0n = in02;
        in1n = in12;
        diagn = diag2;
        haven = more2;
    };
    while (have) {
        step(t0s, t1s);
        if (!have) break;
        step(t1s, t0s);
    }
    // rows 32-63's partial dK / dV are added to rows 0-31's (fixed order) through LDS
    float* red = reinterpret_cast<float*>(tb);   // 4 slots of ND x 16 x 64 floats
    float* slot = red + (2 * half + kh) * (ND * 16 * 64);
    static_assert(2 * TE * 2 >= 4 * ND * 16 * 64 * 4, "reduction space");
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        f32x16* acc = pass == 0 ? dv : dk;
        if (rh == 1)
#pragma unroll
            for (int i = 0; i < ND; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) slot[(i * 16 + r) * 64 + lane] = acc[i][r];
        __syncthreads();
        if (rh == 0)
#pragma unroll
            for (int i = 0; i < ND; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][r] += slot[(i * 16 + r) * 64 + lane];
        __syncthreads();
    }
    if (!live || rh != 0) return;
    float* dkp = a.dk + krow * D;
    float* dvp = a.dv + krow * D;
    const float pt = dz_scale(a.qkvmax + 2, D);   // the tiles give s dV and t s dK
    const float fk = a.scale / (sc * pt * sq), fv = 1.f / sc;
#pragma unroll
    for (int i = 0; i < ND; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f32x4 x, y;
            x.x = dk[i][4 * j + 0] * fk;
            x.y = dk[i][4 * j + 1] * fk;
            x.z = dk[i][4 * j + 2] * fk;
            x.w = dk[i][4 * j + 3] * fk;
            y.x = dv[i][4 * j + 0] * fv;
            y.y = dv[i][4 * j + 1] * fv;
            y.z = dv[i][4 * j + 2] * fv;
            y.w = dv[i][4 * j + 3] * fv;
            *reinterpret_cast<f32x4*>(dkp + 32 * i + 8 * j + 4 * h) = x;
            *reinterpret_cast<f32x4*>(dvp + 32 * i + 8 * j + 4 * h) = y;
        }
}

__device__ __forceinline__ bool dbit(const uint32_t* db, int32_t x) { return (db[x >> 5] >> (x & 31)) & 1u; }

// ------------------------------------------------------------------ column pass
// Work list: chunk = 64 consecutive entries of one head's vertical list.  The
// query blocks that can see a chunk form a suffix of the local blocks (global
// block numbers rise with the local block in both ring layouts), starting at
// the first block whose global number reaches the block of the chunk's
// smallest column plus the head's run of selected block-diagonals from 0
// (nearer query blocks reach every column of the chunk through one of those
// diagonals, i.e. through selected blocks); that suffix is cut into items of
// `span` blocks.  One workgroup builds the list (plain scans, so
// the list and hence the summation order are fixed by the index alone).
constexpr int kPlanThreads = 1024;

// Exclusive prefix sum over the 1024-thread workgroup; tmp holds 17 ints.
__device__ int plan_scan(int v, int* tmp, int* total) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) tmp[wid] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int w = 0; w < kPlanThreads / 64; ++w) {
            const int t = tmp[w];
            tmp[w] = run;
            run += t;
        }
        tmp[16] = run;
    }
    __syncthreads();
    const int res = tmp[wid] + x - v;
    *total = tmp[16];
    __syncthreads();
    return res;
}

__global__ void __launch_bounds__(kPlanThreads) bwd_colplan_kernel(AttnArgs a) {
    __shared__ int tmp[17];
    __shared__ long long part[kPlanThreads / 64];
    if (index_overflowed(a.overflow)) return;   // the column kernels return as well
    const int tid = threadIdx.x;
    const int BH = a.B * a.Hq;
    // chunks per head (entries past the capacity are ignored)
    int carry = 0;
    for (int base = 0; base < BH; base += kPlanThreads) {
        const int h = base + tid;
        int n = 0;
        if (h < BH) {
            const int64_t v0 = min(a.vcol_ptr[h], a.vcol_cap), v1 = min(a.vcol_ptr[h + 1], a.vcol_cap);
            n = v1 > v0 ? int((v1 - v0 + 63) / 64) : 0;
        }
        int tot;
        const int ex = plan_scan(n, tmp, &tot);
        if (h < BH) a.col_choff[h] = carry + ex;
        carry += tot;
    }
    const int nc = carry;
    if (tid == 0) a.col_choff[BH] = nc;
    __syncthreads();
    // per chunk: head, first entry, first candidate query block
    long long cand = 0;
    for (int g = tid; g < nc; g += kPlanThreads) {
        int lo = 0, hi = BH;  // col_choff[lo] <= g < col_choff[hi]
        while (hi - lo > 1) {
            const int m = (lo + hi) >> 1;
            if (a.col_choff[m] <= g) lo = m; else hi = m;
        }
        const int64_t e0 = a.vcol_ptr[lo] + int64_t(g - a.col_choff[lo]) * 64;
        const int32_t cb = min(max(a.vcol_idx[e0], 0), a.Nk - 1) >> 6;
        const int32_t cg = a.k_blk_global[cb];
        // run of selected block-diagonals 0 .. run - 1 of the head: a column
        // of block kc lies on one of them for every query block below kc + run,
        // so no column of the chunk is seen before global block cg + run
        int64_t run = 0;
        const uint32_t* db = a.diag_bits + int64_t(lo) * a.dwords;
        for (int w = 0; w < a.dwords; ++w) {
            const uint32_t word = db[w];
            if (word != 0xffffffffu) {
                run += __builtin_ctz(~word);
                break;
            }
            run += 32;
        }
        const int64_t first = int64_t(cg) + run;
        int L = 0, R = a.nqb;  // first local query block with global block >= cg + run
        while (L < R) {
            const int m = (L + R) >> 1;
            if (a.q_blk_global[m] < first) L = m + 1; else R = m;
        }
        a.col_head[g] = lo;
        a.col_e0[g] = e0;
        a.col_qlo[g] = L;
        cand += a.nqb - L;
    }
    for (int o = 32; o > 0; o >>= 1) cand += __shfl_xor(cand, o);
    if ((tid & 63) == 0) part[tid >> 6] = cand;
    __syncthreads();
    long long total = 0;
    for (int w = 0; w < kPlanThreads / 64; ++w) total += part[w];
    const long long want = (total + a.col_budget - 1) / a.col_budget;
    const int span = int(want > kColMinSpan ? want : kColMinSpan);
    if (tid == 0) a.col_span[0] = span;
    // items per chunk, scanned (chunk g was filled by this same thread above)
    carry = 0;
    for (int base = 0; base < nc; base += kPlanThreads) {
        const int g = base + tid;
        const int n = g < nc ? (a.nqb - a.col_qlo[g] + span - 1) / span : 0;
        int tot;
        const int ex = plan_scan(n, tmp, &tot);
        if (g < nc) a.col_item[g] = carry + ex;
        carry += tot;
    }
    if (tid == 0) a.col_item[nc] = carry;
}

// One workgroup per item: the item's chunk of verticals (64 key rows of one
// query head, held in registers) against each query block of the item that
// sees some of them outside its selected block-diagonals; the partial dK / dV
// of the item go to its own slot (grid = item capacity; surplus workgroups
// exit, consecutive items land on different XCDs).
template <int D>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1))) bwd_dkdv_col_kernel(AttnArgs a) {
    constexpr int KD = D / 16, ND = D / 32;
    // two query-tile buffers and their key limits: the next active tile's
    // loads are in flight while the current one is computed
    __shared__ __attribute__((aligned(16))) uint16_t ts[2][KvTile<D>::kElems];
    __shared__ int32_t clims[2][64];
    if (index_overflowed(a.overflow)) return;   // no work list was planned
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nc = a.col_choff[a.B * a.Hq];
    const int item = int(blockIdx.x);
    if (item >= a.col_item[nc]) return;
    int g = 0, ghi = nc;  // col_item[g] <= item < col_item[ghi]
    while (ghi - g > 1) {
        const int m = (g + ghi) >> 1;
        if (a.col_item[m] <= item) g = m; else ghi = m;
    }
    const int bh = a.col_head[g];
    const int64_t e0 = a.col_e0[g];
    const int64_t v1 = min(a.vcol_ptr[bh + 1], a.vcol_cap);
    const int cnt = int(min<int64_t>(64, v1 - e0));
    const int span = a.col_span[0];
    const int qb0 = a.col_qlo[g] + (item - a.col_item[g]) * span;
    const int qb1 = min(a.nqb, qb0 + span);
    const int b = bh / a.Hq, hq = bh % a.Hq, hk = hq / (a.Hq / a.Hkv);
    const int key = 32 * w + l32;
    const bool valid = key < cnt;
    const int32_t col = min(max(a.vcol_idx[e0 + (valid ? key : 0)], 0), a.Nk - 1);
    const int32_t cg = a.k_blk_global[col >> 6];
    const int32_t cin = col & 63;
    const int64_t krow = (int64_t(b) * a.Hkv + hk) * a.Nk + col;
    u32x4 kreg[KD], vreg[KD];
#pragma unroll
    for (int s = 0; s < KD; ++s) {
        kreg[s] = *reinterpret_cast<const u32x4*>(a.k16 + krow * D + 16 * s + 8 * h);
        vreg[s] = *reinterpret_cast<const u32x4*>(a.v16 + krow * D + 16 * s + 8 * h);
    }
    f32x16 dv[ND], dk[ND];
#pragma unroll
    for (int i = 0; i < ND; ++i) {
        dv[i] = f32x16{};
        dk[i] = f32x16{};
    }
    const float sq = operand_scale(a.qkvmax), sk = operand_scale(a.qkvmax + 1);
    const float isv = dz_scale(a.qkvmax + 2, D) / operand_scale(a.qkvmax + 2);   // t / sv
    const float c2 = a.scale * kLog2e / (sq * sk);
    const float sc = dout_scale(a.dmax);
    const uint32_t* db = a.diag_bits + int64_t(bh) * a.dwords;
    // the next query block from q on where some column of the chunk is not
    // covered by a selected block-diagonal (qb1 if none); its key limits go
    // to clims[buf] and its loads into ts[buf]
    auto next_active = [&](int q, int buf) {
        for (; q < qb1; ++q) {
            const int32_t qg = a.q_blk_global[q];
            const bool active = valid && qg >= cg && !dbit(db, qg - cg);
            if (__syncthreads_or(active)) {
                clims[buf][key] = active ? (qg == cg ? cin : 0) : 64;
                kv_load_query_tile<D, 2>(ts[buf], a, bh, q, w, lane);
                break;
            }
        }
        return q;
    };
    int cur = next_active(qb0, 0), buf = 0;
    wait_vmem();
    __syncthreads();
    while (cur < qb1) {
        const int nxt = next_active(cur + 1, buf ^ 1);
        kv_tile<D, true>(ts[buf], kreg, vreg, clims[buf], key, c2, isv, lane, dv, dk);
        wait_vmem();
        __syncthreads();
        cur = nxt;
        buf ^= 1;
    }
    if (!valid) return;
    const int64_t slot = int64_t(item) * 64 + key;
    float* dkp = a.dk_col + slot * D;
    float* dvp = a.dv_col + slot * D;
    const float pt = dz_scale(a.qkvmax + 2, D);   // the tiles give s dV and t s dK
    const float fk = a.scale / (sc * pt * sq), fv = 1.f / sc;
#pragma unroll
    for (int i = 0; i < ND; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f32x4 x, y;
            x.x = dk[i][4 * g + 0] * fk;
            x.y = dk[i][4 * g + 1] * fk;
            x.z = dk[i][4 * g + 2] * fk;
            x.w = dk[i][4 * g + 3] * fk;
            y.x = dv[i][4 * g + 0] * fv;
            y.y = dv[i][4 * g + 1] * fv;
            y.z = dv[i][4 * g + 2] * fv;
            y.w = dv[i][4 * g + 3] * fv;
            *reinterpret_cast<f32x4*>(dkp + 32 * i + 8 * g + 4 * h) = x;
            *reinterpret_cast<f32x4*>(dvp + 32 * i + 8 * g + 4 * h) = y;
        }
}

// Adds the column partials of key block kb into dK / dV: one workgroup per
// (b, KV head, key block); query heads in order, then each chunk's items in
// order.
// One workgroup per (KV head, 64-key block): for each query head of the group
// in order, the head's vertical entries inside the block (distinct keys, so
// distinct rows) are merged one per wave; the heads follow one another, so
// every row receives its heads' sums in a fixed order.
constexpr int kMergeThreads = 512;
__global__ void __launch_bounds__(kMergeThreads) bwd_colmerge_kernel(AttnArgs a) {
    __shared__ int64_t span_lo[kMergeThreads], span_hi[kMergeThreads];
    if (index_overflowed(a.overflow)) return;   // no work list was planned
    const int BK = a.B * a.Hkv;
    const int bk = int(blockIdx.x % BK);
    const int kb = int(blockIdx.x / BK);
    const int b = bk / a.Hkv, hk = bk % a.Hkv;
    const int G = a.Hq / a.Hkv;
    const int lo = kb * 64, hi = lo + 64;
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    constexpr int NW = kMergeThreads / 64;
    // first entry >= v of an ascending list [L, R)
    auto lower = [&](int64_t L, int64_t R, int32_t v) {
        while (L < R) {
            const int64_t m = (L + R) >> 1;
            if (a.vcol_idx[m] < v) L = m + 1; else R = m;
        }
        return L;
    };
    for (int gb = 0; gb < G; gb += kMergeThreads) {
        const int ng = min(kMergeThreads, G - gb);
        if (int(threadIdx.x) < ng) {   // one thread per head: the head's entries in this block
            const int bh = b * a.Hq + hk * G + gb + threadIdx.x;
            const int64_t v0 = a.vcol_ptr[bh], v1 = min(a.vcol_ptr[bh + 1], a.vcol_cap);
            const int64_t L = v0 < v1 ? lower(v0, v1, lo) : v1;
            span_lo[threadIdx.x] = L;
            span_hi[threadIdx.x] = L < v1 ? lower(L, v1, hi) : L;
        }
        __syncthreads();
        for (int gi = 0; gi < ng; ++gi) {
            const int bh = b * a.Hq + hk * G + gb + gi;
            const int64_t v0 = a.vcol_ptr[bh];
            const int32_t c0 = a.col_choff[bh];
            for (int64_t e = span_lo[gi] + w; e < span_hi[gi]; e += NW) {
                const int64_t ch = c0 + (e - v0) / 64;
                const int key = int((e - v0) % 64);
                const int i0 = a.col_item[ch], i1 = a.col_item[ch + 1];
                const int64_t row = int64_t(bk) * a.Nk + a.vcol_idx[e];
                for (int j = lane; j < a.d; j += 64) {
                    // four independent partial sums (eight loads in flight),
                    // combined in a fixed order
                    float sk[4] = {0.f, 0.f, 0.f, 0.f}, sv[4] = {0.f, 0.f, 0.f, 0.f};
                    int it = i0;
                    for (; it + 4 <= i1; it += 4) {
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            sk[u] += a.dk_col[(int64_t(it + u) * 64 + key) * a.d + j];
                            sv[u] += a.dv_col[(int64_t(it + u) * 64 + key) * a.d + j];
                        }
                    }
                    for (; it < i1; ++it) {
                        sk[0] += a.dk_col[(int64_t(it) * 64 + key) * a.d + j];
                        sv[0] += a.dv_col[(int64_t(it) * 64 + key) * a.d + j];
                    }
                    a.dk[row * a.d + j] += (sk[0] + sk[1]) + (sk[2] + sk[3]);
                    a.dv[row * a.d + j] += (sv[0] + sv[1]) + (sv[2] + sv[3]);
                }
            }
            __syncthreads();   // the next head may add to the same rows
        }
    }
}

template <int D>
hipError_t launch_bwd_d(const AttnArgs& a, hipStream_t s) {
    const int64_t rows = int64_t(a.B) * a.Hq * a.Nq;
    { TraceScope _t("bwd_init", s); hipLaunchKernelGGL(bwd_init_kernel, dim3(1), dim3(64), 0, s, a); }
    // Q-side data (Delta, lse rows, max |dO|, max |Q|, the Q and dO copies) is
    // the same for every ring step of a worker: a later step may reuse it
    const bool qside = !a.reuse_qrows;
    if (qside && rows > 0) {
        TraceScope _t("bwd_delta", s);
        const int64_t groups = (rows + 127) / 128;
        const dim3 grid(unsigned(groups < kDeltaBlocks ? groups : int64_t(kDeltaBlocks)));
        if (a.o_f32)
            hipLaunchKernelGGL((bwd_delta_kernel<D / 16, true>), grid, dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((bwd_delta_kernel<D / 16, false>), grid, dim3(256), 0, s, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // scaled fp16 copies: Q, K, V to max in [2^14, 2^15), dO to [8, 16)
    const int64_t nkv = int64_t(a.B) * a.Hkv * a.Nk * a.d;
    const int64_t nq = int64_t(a.B) * a.Hq * a.Nq * a.d;
    if (qside && (e = launch_absmax(a.q, nq, a.qkvmax, s)) != hipSuccess) return e;
    if ((e = launch_absmax(a.k, nkv, a.qkvmax + 1, s)) != hipSuccess) return e;
    if ((e = launch_absmax(a.v, nkv, a.qkvmax + 2, s)) != hipSuccess) return e;
    // row values after max |V| (the probability scale t)
    if (rows > 0) {
        TraceScope _t("bwd_rowprep", s);
        const int64_t want = (rows + 255) / 256;
        hipLaunchKernelGGL(bwd_rowprep_kernel, dim3(unsigned(want < kDeltaBlocks ? want : int64_t(kDeltaBlocks))),
                           dim3(256), 0, s, a);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (qside && (e = launch_to_f16(a.q, a.q16, nq, a.qkvmax, kOperandExp, s)) != hipSuccess) return e;
    if ((e = launch_to_f16(a.k, a.k16, nkv, a.qkvmax + 1, kOperandExp, s)) != hipSuccess) return e;
    if ((e = launch_to_f16(a.v, a.v16, nkv, a.qkvmax + 2, kOperandExp, s)) != hipSuccess) return e;
    if (qside && (e = launch_to_f16(a.dout, a.g16, nq, a.dmax, 4, s)) != hipSuccess) return e;
    const int64_t qgrid = int64_t(a.B) * a.Hq * ((a.nqb + 1) / 2);
    if (qgrid > 0) { TraceScope _t("bwd_dq", s); hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3(unsigned(qgrid)), dim3(kDqThreads), 0, s, a); }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t kpgrid = int64_t(a.B) * a.Hkv * ((a.nkb + 1) / 2);
    if (kpgrid > 0) {
        TraceScope _t("bwd_dkdv", s);
        hipLaunchKernelGGL(bwd_dkdv_rows_kernel<D>, dim3(unsigned(kpgrid)), dim3(kKvRowsThreads), 0, s, a);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    { TraceScope _t("bwd_colplan", s); hipLaunchKernelGGL(bwd_colplan_kernel, dim3(1), dim3(kPlanThreads), 0, s, a); }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (a.col_slots > 0) {
        TraceScope _t("bwd_dkdv_col", s);
        hipLaunchKernelGGL(bwd_dkdv_col_kernel<D>, dim3(unsigned(a.col_slots)), dim3(kThreads), 0, s, a);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t kgrid = int64_t(a.B) * a.Hkv * a.nkb;
    if (kgrid > 0) { TraceScope _t("bwd_colmerge", s); hipLaunchKernelGGL(bwd_colmerge_kernel, dim3(unsigned(kgrid)), dim3(kMergeThreads), 0, s, a); }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd(const AttnArgs& a, hipStream_t s) {
    return a.d == 128 ? launch_bwd_d<128>(a, s) : launch_bwd_d<64>(a, s);
}

}  // namespace msparse
