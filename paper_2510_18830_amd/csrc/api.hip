// C ABI of libmsparse: argument validation, workspace carve-up and launches.
// Every check runs on the host before the first launch, so an error return
// leaves the stream untouched.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <string>

#include "common.h"
#include "kernels.h"

using namespace msparse;

namespace {

thread_local std::string g_last_error;

msparse_status fail(msparse_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

// Every tensor named in the header's conventions is read or written with
// 16-byte vector accesses; NULL (an optional tensor) passes.
bool misaligned(std::initializer_list<const void*> ps) {
    for (const void* p : ps)
        if (reinterpret_cast<uintptr_t>(p) & 15u) return true;
    return false;
}

bool sync_check_enabled() {
    static int v = [] {
        const char* e = getenv("MSPARSE_SYNC_CHECK");
        return (e && e[0] && e[0] != '0') ? 1 : 0;
    }();
    return v != 0;
}

msparse_status check_hip(hipError_t e, hipStream_t s, const char* what) {
    if (e != hipSuccess) return fail(MSPARSE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    if (sync_check_enabled()) {
        // a stream under graph capture cannot be synchronised: its work runs
        // at replay, so the check is skipped there
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        e = hipStreamIsCapturing(s, &cap);
        if (e == hipSuccess && cap == hipStreamCaptureStatusNone) e = hipStreamSynchronize(s);
        if (e == hipSuccess) e = hipGetLastError();
        if (e != hipSuccess) return fail(MSPARSE_ERR_HIP, "%s (sync check): %s", what, hipGetErrorString(e));
    }
    return MSPARSE_OK;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Bump allocator over the caller's workspace.
struct Carve {
    char* base;
    size_t off = 0;
    template <class T>
    T* take(size_t count) {
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off = align_up(off + count * sizeof(T));
        return p;
    }
};

float resolve_scale(const msparse_dims* d) { return d->scale > 0.f ? d->scale : 1.0f / std::sqrt(float(d->head_dim)); }

msparse_status check_dims(const msparse_dims* d, bool same_len) {
    if (!d) return fail(MSPARSE_ERR_INVALID, "dims is NULL");
    if (d->batch < 1 || d->heads_q < 1 || d->heads_kv < 1 || d->seq_q < 0 || d->seq_k < 0)
        return fail(MSPARSE_ERR_INVALID, "batch, heads must be >= 1 and lengths >= 0");
    if (d->heads_q % d->heads_kv != 0)
        return fail(MSPARSE_ERR_INVALID, "heads_q (%d) is not a multiple of heads_kv (%d)", d->heads_q, d->heads_kv);
    if (d->head_dim != 64 && d->head_dim != 128)
        return fail(MSPARSE_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", d->head_dim);
    if (d->block != kBlock) return fail(MSPARSE_ERR_UNSUPPORTED, "block %d (supported: 64)", d->block);
    if (d->causal != 1) return fail(MSPARSE_ERR_UNSUPPORTED, "only causal attention is supported");
    if (d->seq_q % kBlock || d->seq_k % kBlock)
        return fail(MSPARSE_ERR_UNSUPPORTED, "sequence lengths (%d, %d) must be multiples of 64", d->seq_q, d->seq_k);
    if (same_len && d->seq_q != d->seq_k) return fail(MSPARSE_ERR_INVALID, "seq_q != seq_k");
    if (!std::isfinite(d->scale)) return fail(MSPARSE_ERR_INVALID, "scale is not finite");
    const int64_t big = int64_t(d->batch) * d->heads_q * int64_t(std::max(d->seq_q, d->seq_k));
    if (big > (int64_t(1) << 31) - 1) return fail(MSPARSE_ERR_UNSUPPORTED, "batch * heads * seq exceeds 2^31 rows");
    return MSPARSE_OK;
}

struct RingInfo {
    int32_t world = 1, rank = 0, step = 0, layout = MSPARSE_LAYOUT_STRIPED, shard = 0;
};

// Shard held by `rank` at `step`: flat ring, or the hierarchical order of
// Algorithm 2 (outer ring over nodes of `inner` cards, inner ring per node).
int32_t ring_shard(int32_t world, int32_t inner, int32_t rank, int32_t step) {
    if (world < 1 || rank < 0 || rank >= world || step < 0 || step >= world) return -1;
    if (inner < 0 || (inner > 0 && world % inner != 0)) return -1;
    if (inner <= 1 || inner == world) return ((rank - step) % world + world) % world;
    const int32_t nodes = world / inner;
    const int32_t node = rank / inner, card = rank % inner;
    const int32_t i = step / inner, j = step % inner;
    return ((node - i) % nodes + nodes) % nodes * inner + ((card - j) % inner + inner) % inner;
}

msparse_status check_ring(const msparse_dims* d, const msparse_ring* r, RingInfo* out) {
    RingInfo ri;
    if (r) {
        if (r->world < 1 || r->rank < 0 || r->rank >= r->world || r->step < 0 || r->step >= r->world)
            return fail(MSPARSE_ERR_INVALID, "ring world %d rank %d step %d", r->world, r->rank, r->step);
        if (r->layout != MSPARSE_LAYOUT_STRIPED && r->layout != MSPARSE_LAYOUT_ZIGZAG)
            return fail(MSPARSE_ERR_INVALID, "ring layout %d", r->layout);
        if (r->inner < 0 || (r->inner > 0 && r->world % r->inner != 0))
            return fail(MSPARSE_ERR_INVALID, "ring inner %d does not divide world %d", r->inner, r->world);
        ri.world = r->world;
        ri.rank = r->rank;
        ri.step = r->step;
        ri.layout = r->layout;
        ri.shard = ring_shard(r->world, r->inner, r->rank, r->step);
        if (r->layout == MSPARSE_LAYOUT_ZIGZAG && (d->seq_q / kBlock) % 2 != 0)
            return fail(MSPARSE_ERR_UNSUPPORTED, "zigzag shards need an even number of 64-token blocks");
    }
    if (d->seq_q != d->seq_k) return fail(MSPARSE_ERR_INVALID, "query and KV shards must have equal length");
    const int64_t ng = int64_t(d->seq_q) * ri.world;
    if (ng > (int64_t(1) << 30)) return fail(MSPARSE_ERR_UNSUPPORTED, "global sequence too long");
    *out = ri;
    return MSPARSE_OK;
}

// ------------------------------------------------------------------ index
struct IndexPlan {
    IndexArgs a{};
    size_t bytes = 0;
};

IndexPlan plan_index(const msparse_dims* d, int32_t k_v, int32_t k_s, const RingInfo& ri, void* ws,
                     bool own_ptrs) {
    IndexPlan p;
    IndexArgs& a = p.a;
    a.BH = d->batch * d->heads_q;
    a.k_v = k_v;
    a.k_s = k_s;
    a.nqb = d->seq_q / kBlock;
    a.nkb = d->seq_k / kBlock;
    a.nb = a.nqb * ri.world;
    a.world = ri.world;
    a.rank = ri.rank;
    a.shard = ri.shard;
    a.layout = ri.layout;
    const int64_t ng = int64_t(a.nb) * kBlock;
    a.vwords = int32_t((ng + 31) / 32);
    a.dwords = (a.nb + 31) / 32;
    Carve c{static_cast<char*>(ws)};
    a.vbits = c.take<uint32_t>(size_t(a.BH) * a.vwords);
    a.vlist = c.take<int32_t>(size_t(a.BH) * k_v);
    a.vcnt = c.take<int32_t>(a.BH);
    a.dlist = c.take<int32_t>(size_t(a.BH) * a.nb);
    a.dcnt = c.take<int32_t>(a.BH);
    a.dbits = c.take<uint32_t>(size_t(a.BH) * a.dwords);
    a.dpre = c.take<int32_t>(size_t(a.BH) * (a.dwords + 1));
    a.cumv = c.take<int32_t>(size_t(a.BH) * (a.nb + 1));
    a.drun = c.take<int32_t>(a.BH);
    a.cnt_blk = c.take<int64_t>(size_t(a.BH) * a.nqb);
    a.cnt_col = c.take<int64_t>(size_t(a.BH) * a.nqb);
    a.cnt_kblk = c.take<int64_t>(size_t(a.BH) * a.nkb);
    a.cnt_vcol = c.take<int64_t>(a.BH);
    {
        const int64_t nmax = std::max<int64_t>(int64_t(a.BH) * std::max(a.nqb, a.nkb), a.BH);
        a.scan_stride = (nmax + kScanEntriesPerBlock - 1) / kScanEntriesPerBlock;
        a.scan_sums = c.take<int64_t>(size_t(4 * a.scan_stride));
    }
    if (own_ptrs) {
        a.blk_ptr = c.take<int64_t>(size_t(a.BH) * a.nqb + 1);
        a.col_ptr = c.take<int64_t>(size_t(a.BH) * a.nqb + 1);
        a.kblk_ptr = c.take<int64_t>(size_t(a.BH) * a.nkb + 1);
        a.vcol_ptr = c.take<int64_t>(size_t(a.BH) + 1);
    } else {
        // room for the pointer arrays is reserved either way so the size query
        // does not depend on the mode
        c.take<int64_t>(size_t(a.BH) * a.nqb + 1);
        c.take<int64_t>(size_t(a.BH) * a.nqb + 1);
        c.take<int64_t>(size_t(a.BH) * a.nkb + 1);
        c.take<int64_t>(size_t(a.BH) + 1);
    }
    p.bytes = c.off;
    return p;
}

msparse_status check_index_inputs(const msparse_dims* d, const int32_t* v_idx, int32_t k_v, const int32_t* s_idx,
                                  int32_t k_s, const msparse_ring* ring, RingInfo* ri) {
    msparse_status st = check_dims(d, false);
    if (st) return st;
    if ((st = check_ring(d, ring, ri))) return st;
    if (!v_idx || !s_idx) return fail(MSPARSE_ERR_INVALID, "v_idx / s_idx is NULL");
    const int64_t ng = int64_t(d->seq_q) * ri->world;
    if (k_v < 1 || k_v > ng || k_s < 1 || k_s > ng)
        return fail(MSPARSE_ERR_INVALID, "budgets k_v=%d k_s=%d outside [1, %lld]", k_v, k_s, (long long)ng);
    if (d->seq_q == 0) return fail(MSPARSE_ERR_INVALID, "empty sequence");
    const int64_t items = int64_t(d->batch) * d->heads_q * std::max(d->seq_q, d->seq_k) / kBlock;
    if (items > int64_t(kScanEntriesPerBlock) * kScanEntriesPerBlock)
        return fail(MSPARSE_ERR_UNSUPPORTED, "%lld (head, block) items exceed the index scan's %d^2",
                    (long long)items, kScanEntriesPerBlock);
    return MSPARSE_OK;
}

msparse_status check_index_struct(const msparse_dims* d, const msparse_index* x, bool need_transpose) {
    if (!x) return fail(MSPARSE_ERR_INVALID, "index is NULL");
    if (!x->blk_ptr || !x->col_ptr || !x->q_blk_global || !x->k_blk_global || !x->diag_bits)
        return fail(MSPARSE_ERR_INVALID, "index arrays are NULL");
    if ((x->blk_cap > 0 && !x->blk_idx) || (x->col_cap > 0 && !x->col_idx))
        return fail(MSPARSE_ERR_INVALID, "index entry arrays are NULL");
    if (need_transpose && (!x->kblk_ptr || !x->vcol_ptr || (x->blk_cap > 0 && !x->kblk_idx) ||
                           (x->vcol_cap > 0 && !x->vcol_idx)))
        return fail(MSPARSE_ERR_INVALID, "transposed index arrays are NULL");
    if (x->blk_cap < 0 || x->col_cap < 0 || x->vcol_cap < 0) return fail(MSPARSE_ERR_INVALID, "negative capacity");
    if (x->world < 1) return fail(MSPARSE_ERR_INVALID, "index world %d < 1", x->world);
    (void)d;
    return MSPARSE_OK;
}

// ------------------------------------------------------------------ allocation-free index build
// Scratch of msparse_build_index_noalloc: file-scope device memory, one copy
// per GPU, made when the code object loads on that GPU and held until the
// process ends.  In host code `scratch` names a host-side stand-in, not a
// device address: the address each GPU uses comes from hipGetSymbolAddress
// (scratch_on_current_device) and is the only one passed to kernels.
constexpr size_t kNoallocScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 256;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up once per device (with
// that device current) and kept.
msparse_status scratch_on_current_device(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(MSPARSE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return fail(MSPARSE_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(MSPARSE_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return MSPARSE_OK;
}

}  // namespace

extern "C" {

const char* msparse_strerror(msparse_status s) {
    switch (s) {
        case MSPARSE_OK: return "ok";
        case MSPARSE_ERR_INVALID: return "invalid argument";
        case MSPARSE_ERR_UNSUPPORTED: return "unsupported configuration";
        case MSPARSE_ERR_CAPACITY: return "index capacity too small";
        case MSPARSE_ERR_WORKSPACE: return "workspace too small";
        case MSPARSE_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char* msparse_last_error(void) { return g_last_error.c_str(); }

int32_t msparse_ring_shard(int32_t world, int32_t inner, int32_t rank, int32_t step) {
    return ring_shard(world, inner, rank, step);
}

// ------------------------------------------------------------------ index
size_t msparse_index_workspace(const msparse_dims* dims, int32_t k_v, int32_t k_s, const msparse_ring* ring) {
    RingInfo ri;
    if (check_dims(dims, false) || check_ring(dims, ring, &ri) || k_v < 1 || k_s < 1) return 0;
    return plan_index(dims, k_v, k_s, ri, nullptr, true).bytes;
}

msparse_status msparse_index_count(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v, const int32_t* s_idx,
                                   int32_t k_s, const msparse_ring* ring, int64_t* blk_nnz, int64_t* col_nnz,
                                   int64_t* vcol_nnz, void* ws, size_t ws_bytes, void* stream) {
    RingInfo ri;
    msparse_status st = check_index_inputs(dims, v_idx, k_v, s_idx, k_s, ring, &ri);
    if (st) return st;
    if (!blk_nnz || !col_nnz || !vcol_nnz) return fail(MSPARSE_ERR_INVALID, "count outputs are NULL");
    IndexPlan p = plan_index(dims, k_v, k_s, ri, ws, true);
    if (!ws || ws_bytes < p.bytes)
        return fail(MSPARSE_ERR_WORKSPACE, "index workspace %zu < %zu bytes", ws_bytes, p.bytes);
    p.a.v_idx = v_idx;
    p.a.s_idx = s_idx;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_hip(launch_index_prep(p.a, s), s, "index prep"))) return st;
    if ((st = check_hip(launch_index_count(p.a, s), s, "index count"))) return st;
    if ((st = check_hip(launch_index_scan(p.a, s), s, "index scan"))) return st;
    int64_t tot[3];
    const int64_t nq = int64_t(p.a.BH) * p.a.nqb;
    hipError_t e = hipMemcpyAsync(&tot[0], p.a.blk_ptr + nq, 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&tot[1], p.a.col_ptr + nq, 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&tot[2], p.a.vcol_ptr + p.a.BH, 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(MSPARSE_ERR_HIP, "index count readback: %s", hipGetErrorString(e));
    *blk_nnz = tot[0];
    *col_nnz = tot[1];
    *vcol_nnz = tot[2];
    return MSPARSE_OK;
}

msparse_status msparse_build_index(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v, const int32_t* s_idx,
                                   int32_t k_s, const msparse_ring* ring, const msparse_index* index, void* ws,
                                   size_t ws_bytes, void* stream) {
    RingInfo ri;
    msparse_status st = check_index_inputs(dims, v_idx, k_v, s_idx, k_s, ring, &ri);
    if (st) return st;
    if ((st = check_index_struct(dims, index, true))) return st;
    if (index->world != ri.world)
        return fail(MSPARSE_ERR_INVALID, "index world %d differs from the ring world %d", index->world, ri.world);
    IndexPlan p = plan_index(dims, k_v, k_s, ri, ws, false);
    if (!ws || ws_bytes < p.bytes)
        return fail(MSPARSE_ERR_WORKSPACE, "index workspace %zu < %zu bytes", ws_bytes, p.bytes);
    // Without an overflow flag the capacities must cover the worst case.
    const int64_t BH = p.a.BH, nqb = p.a.nqb, nkb = p.a.nkb;
    const int64_t dmax = std::min<int64_t>(p.a.nb, 2 * int64_t(k_s));
    const int64_t blk_bound = BH * nqb * std::min<int64_t>(nkb, dmax);
    const int64_t col_bound = BH * nqb * std::min<int64_t>(k_v, nkb * kBlock);
    const int64_t vcol_bound = BH * std::min<int64_t>(k_v, nkb * kBlock);
    if (!index->overflow && (index->blk_cap < blk_bound || index->col_cap < col_bound || index->vcol_cap < vcol_bound))
        return fail(MSPARSE_ERR_CAPACITY,
                    "capacities (%lld, %lld, %lld) below the worst case (%lld, %lld, %lld) and no overflow flag",
                    (long long)index->blk_cap, (long long)index->col_cap, (long long)index->vcol_cap,
                    (long long)blk_bound, (long long)col_bound, (long long)vcol_bound);
    IndexArgs& a = p.a;
    a.v_idx = v_idx;
    a.s_idx = s_idx;
    a.blk_ptr = index->blk_ptr;
    a.col_ptr = index->col_ptr;
    a.kblk_ptr = index->kblk_ptr;
    a.vcol_ptr = index->vcol_ptr;
    a.blk_idx = index->blk_idx;
    a.blk_cap = index->blk_cap;
    a.col_idx = index->col_idx;
    a.col_cap = index->col_cap;
    a.kblk_idx = index->kblk_idx;
    a.vcol_idx = index->vcol_idx;
    a.vcol_cap = index->vcol_cap;
    a.diag_bits_out = index->diag_bits;
    a.q_blk_global = index->q_blk_global;
    a.k_blk_global = index->k_blk_global;
    a.overflow = index->overflow;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_hip(launch_index_prep(a, s), s, "index prep"))) return st;   // also clears the overflow flag
    if ((st = check_hip(launch_index_count(a, s), s, "index count"))) return st;
    if ((st = check_hip(launch_index_scan(a, s), s, "index scan"))) return st;
    return check_hip(launch_index_fill(a, s), s, "index fill");
}

msparse_status msparse_index_count_build(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v,
                                         const int32_t* s_idx, int32_t k_s, const msparse_ring* ring,
                                         const msparse_index* index, int64_t* blk_nnz, int64_t* col_nnz,
                                         int64_t* vcol_nnz, void* ws, size_t ws_bytes, void* stream) {
    RingInfo ri;
    msparse_status st = check_index_inputs(dims, v_idx, k_v, s_idx, k_s, ring, &ri);
    if (st) return st;
    if ((st = check_index_struct(dims, index, true))) return st;
    if (!blk_nnz || !col_nnz || !vcol_nnz) return fail(MSPARSE_ERR_INVALID, "count outputs are NULL");
    if (!index->overflow) return fail(MSPARSE_ERR_INVALID, "msparse_index_count_build needs an overflow flag");
    if (index->world != ri.world)
        return fail(MSPARSE_ERR_INVALID, "index world %d differs from the ring world %d", index->world, ri.world);
    IndexPlan p = plan_index(dims, k_v, k_s, ri, ws, false);
    if (!ws || ws_bytes < p.bytes)
        return fail(MSPARSE_ERR_WORKSPACE, "index workspace %zu < %zu bytes", ws_bytes, p.bytes);
    IndexArgs& a = p.a;
    a.v_idx = v_idx;
    a.s_idx = s_idx;
    a.blk_ptr = index->blk_ptr;
    a.col_ptr = index->col_ptr;
    a.kblk_ptr = index->kblk_ptr;
    a.vcol_ptr = index->vcol_ptr;
    a.blk_idx = index->blk_idx;
    a.blk_cap = index->blk_cap;
    a.col_idx = index->col_idx;
    a.col_cap = index->col_cap;
    a.kblk_idx = index->kblk_idx;
    a.vcol_idx = index->vcol_idx;
    a.vcol_cap = index->vcol_cap;
    a.diag_bits_out = index->diag_bits;
    a.q_blk_global = index->q_blk_global;
    a.k_blk_global = index->k_blk_global;
    a.overflow = index->overflow;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_hip(launch_index_prep(a, s), s, "index prep"))) return st;   // also clears the overflow flag
    if ((st = check_hip(launch_index_count(a, s), s, "index count"))) return st;
    if ((st = check_hip(launch_index_scan(a, s), s, "index scan"))) return st;
    int64_t tot[3];
    const int64_t nq = int64_t(a.BH) * a.nqb;
    hipError_t e = hipMemcpyAsync(&tot[0], a.blk_ptr + nq, 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&tot[1], a.col_ptr + nq, 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&tot[2], a.vcol_ptr + a.BH, 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(MSPARSE_ERR_HIP, "index count readback: %s", hipGetErrorString(e));
    *blk_nnz = tot[0];
    *col_nnz = tot[1];
    *vcol_nnz = tot[2];
    if (tot[0] > index->blk_cap || tot[1] > index->col_cap || tot[2] > index->vcol_cap) {
        // the lists stay unfilled: flag the index so that no attention call walks it
        if ((st = check_hip(launch_index_mark_overflow(a, s), s, "index overflow mark"))) return st;
        return fail(MSPARSE_ERR_CAPACITY, "index needs (%lld, %lld, %lld) entries; capacities (%lld, %lld, %lld)",
                    (long long)tot[0], (long long)tot[1], (long long)tot[2], (long long)index->blk_cap,
                    (long long)index->col_cap, (long long)index->vcol_cap);
    }
    return check_hip(launch_index_fill(a, s), s, "index fill");
}

msparse_status msparse_build_index_noalloc(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v,
                                           const int32_t* s_idx, int32_t k_s, const msparse_ring* ring,
                                           const msparse_index* index, void* stream) {
    RingInfo ri;
    msparse_status st = check_index_inputs(dims, v_idx, k_v, s_idx, k_s, ring, &ri);
    if (st) return st;
    if ((st = check_index_struct(dims, index, true))) return st;
    const size_t need = plan_index(dims, k_v, k_s, ri, nullptr, false).bytes;
    if (need > kNoallocScratchBytes)
        return fail(MSPARSE_ERR_WORKSPACE, "index build needs %zu bytes of scratch; the fixed scratch holds %zu",
                    need, kNoallocScratchBytes);
    void* ws = nullptr;
    if ((st = scratch_on_current_device(&ws))) return st;
    return msparse_build_index(dims, v_idx, k_v, s_idx, k_s, ring, index, ws, need, stream);
}

// ------------------------------------------------------------------ attention
static msparse_status fill_attn(const msparse_dims* d, const msparse_index* x, AttnArgs* a) {
    a->B = d->batch;
    a->Hq = d->heads_q;
    a->Hkv = d->heads_kv;
    a->Nq = d->seq_q;
    a->Nk = d->seq_k;
    a->d = d->head_dim;
    a->nqb = d->seq_q / kBlock;
    a->nkb = d->seq_k / kBlock;
    a->scale = resolve_scale(d);
    a->blk_ptr = x->blk_ptr;
    a->blk_idx = x->blk_idx;
    a->col_ptr = x->col_ptr;
    a->col_idx = x->col_idx;
    a->kblk_ptr = x->kblk_ptr;
    a->kblk_idx = x->kblk_idx;
    a->vcol_ptr = x->vcol_ptr;
    a->vcol_idx = x->vcol_idx;
    a->diag_bits = x->diag_bits;
    a->dwords = (d->seq_q / kBlock * x->world + 31) / 32;
    a->q_blk_global = x->q_blk_global;
    a->k_blk_global = x->k_blk_global;
    a->overflow = x->overflow;
    return MSPARSE_OK;
}

// Forward workspace: the scaled fp16 copy of V and the max words.
static size_t carve_fwd(const msparse_dims* d, char* base, AttnArgs* a) {
    Carve c{base};
    uint16_t* v16 = c.take<uint16_t>(size_t(d->batch) * d->heads_kv * d->seq_k * d->head_dim);
    uint32_t* mx = c.take<uint32_t>(3);
    if (a) {
        a->v16 = v16;
        a->qkvmax = mx;
    }
    return c.off;
}

size_t msparse_attn_fwd_workspace(const msparse_dims* dims) {
    if (check_dims(dims, false)) return 0;
    return carve_fwd(dims, nullptr, nullptr);
}

msparse_status msparse_attn_fwd(const msparse_dims* dims, const void* q, const void* k, const void* v,
                                const msparse_index* index, void* out, float* lse, float* out_f32, void* ws,
                                size_t ws_bytes, void* stream) {
    msparse_status st = check_dims(dims, false);
    if (st) return st;
    if (!q || !k || !v || (!out && !out_f32) || !lse) return fail(MSPARSE_ERR_INVALID, "tensor pointer is NULL");
    if (misaligned({q, k, v, out, out_f32, lse})) return fail(MSPARSE_ERR_INVALID, "tensor not 16-byte aligned");
    if ((st = check_index_struct(dims, index, false))) return st;
    const size_t need = msparse_attn_fwd_workspace(dims);
    if (need && (!ws || ws_bytes < need))
        return fail(MSPARSE_ERR_WORKSPACE, "fwd workspace %zu < %zu bytes", ws_bytes, need);
    if (dims->seq_q == 0) return MSPARSE_OK;
    AttnArgs a{};
    fill_attn(dims, index, &a);
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.out = static_cast<uint16_t*>(out);
    a.out_f32 = out_f32;
    a.lse = lse;
    carve_fwd(dims, static_cast<char*>(ws), &a);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return check_hip(launch_attn_fwd(a, s), s, "attn fwd");
}

msparse_status msparse_attn_fwd_merge(const msparse_dims* dims, const void* q, const void* k, const void* v,
                                      const msparse_index* index, float* o_acc, float* lse_acc, void* out_bf16,
                                      int32_t first, void* ws, size_t ws_bytes, void* stream) {
    msparse_status st = check_dims(dims, false);
    if (st) return st;
    if (!q || !k || !v || !o_acc || !lse_acc) return fail(MSPARSE_ERR_INVALID, "tensor pointer is NULL");
    if (misaligned({q, k, v, o_acc, lse_acc, out_bf16}))
        return fail(MSPARSE_ERR_INVALID, "tensor not 16-byte aligned");
    if ((st = check_index_struct(dims, index, false))) return st;
    const size_t need = msparse_attn_fwd_workspace(dims);
    if (need && (!ws || ws_bytes < need))
        return fail(MSPARSE_ERR_WORKSPACE, "fwd workspace %zu < %zu bytes", ws_bytes, need);
    if (dims->seq_q == 0) return MSPARSE_OK;
    AttnArgs a{};
    fill_attn(dims, index, &a);
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.out = static_cast<uint16_t*>(out_bf16);
    a.out_f32 = o_acc;
    a.lse = lse_acc;
    a.merge_acc = first ? 0 : 1;
    carve_fwd(dims, static_cast<char*>(ws), &a);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return check_hip(launch_attn_fwd(a, s), s, "attn fwd merge");
}

msparse_status msparse_merge_out_lse(const msparse_dims* dims, const float* o_part, const float* lse_part, float* o_acc,
                                     float* lse_acc, void* out_bf16, int32_t first, void* stream) {
    msparse_status st = check_dims(dims, false);
    if (st) return st;
    if (!o_part || !lse_part || !o_acc || !lse_acc) return fail(MSPARSE_ERR_INVALID, "tensor pointer is NULL");
    if (misaligned({o_part, lse_part, o_acc, lse_acc, out_bf16}))
        return fail(MSPARSE_ERR_INVALID, "tensor not 16-byte aligned");
    if (dims->seq_q == 0) return MSPARSE_OK;
    MergeArgs m{};
    m.o_part = o_part;
    m.lse_part = lse_part;
    m.o_acc = o_acc;
    m.lse_acc = lse_acc;
    m.out = static_cast<uint16_t*>(out_bf16);
    m.first = first;
    m.rows = int64_t(dims->batch) * dims->heads_q * dims->seq_q;
    m.d = dims->head_dim;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return check_hip(launch_merge(m, s), s, "merge out/lse");
}

// Backward workspace: scaled fp16 copies of K, V, Q and dO, Delta, s Delta, lse2, the
// max words, the column work list and the per-item column partials.
static size_t carve_bwd(const msparse_dims* d, int64_t vcol_cap, char* base, AttnArgs* a) {
    const int64_t bh = int64_t(d->batch) * d->heads_q;
    const ColPlanSizes z = col_plan_sizes(bh, vcol_cap, d->seq_q / kBlock);
    Carve c{base};
    uint16_t* k16 = c.take<uint16_t>(size_t(d->batch) * d->heads_kv * d->seq_k * d->head_dim);
    uint16_t* v16 = c.take<uint16_t>(size_t(d->batch) * d->heads_kv * d->seq_k * d->head_dim);
    uint16_t* q16 = c.take<uint16_t>(size_t(bh) * d->seq_q * d->head_dim);
    uint16_t* g16 = c.take<uint16_t>(size_t(bh) * d->seq_q * d->head_dim);
    float* draw = c.take<float>(size_t(bh) * d->seq_q);
    float* delta = c.take<float>(size_t(bh) * d->seq_q);
    float* lse2 = c.take<float>(size_t(bh) * d->seq_q);
    uint32_t* dmax = c.take<uint32_t>(4);   // max |dO|, |Q|, |K|, |V|
    int32_t* choff = c.take<int32_t>(size_t(bh) + 1);
    int64_t* e0 = c.take<int64_t>(size_t(z.chunk_cap));
    int32_t* head = c.take<int32_t>(size_t(z.chunk_cap));
    int32_t* qlo = c.take<int32_t>(size_t(z.chunk_cap));
    int32_t* item = c.take<int32_t>(size_t(z.chunk_cap) + 1);
    int32_t* span = c.take<int32_t>(1);
    float* dkc = c.take<float>(size_t(z.slots) * kBlock * d->head_dim);
    float* dvc = c.take<float>(size_t(z.slots) * kBlock * d->head_dim);
    if (a) {
        a->k16 = k16;
        a->v16 = v16;
        a->q16 = q16;
        a->g16 = g16;
        a->draw = draw;
        a->delta = delta;
        a->lse2 = lse2;
        a->dmax = dmax;
        a->qkvmax = dmax + 1;
        a->col_choff = choff;
        a->col_e0 = e0;
        a->col_head = head;
        a->col_qlo = qlo;
        a->col_item = item;
        a->col_span = span;
        a->col_chunk_cap = z.chunk_cap;
        a->col_budget = z.budget;
        a->col_slots = z.slots;
        a->dk_col = dkc;
        a->dv_col = dvc;
    }
    return c.off;
}

size_t msparse_attn_bwd_workspace(const msparse_dims* dims, int64_t vcol_cap) {
    if (check_dims(dims, false) || vcol_cap < 0) return 0;
    return carve_bwd(dims, vcol_cap, nullptr, nullptr);
}

msparse_status msparse_attn_bwd(const msparse_dims* dims, const void* q, const void* k, const void* v,
                                const void* out, const float* out_f32, const void* dout, const float* lse,
                                const msparse_index* index, float* dq, float* dk, float* dv, int32_t flags,
                                void* ws, size_t ws_bytes, void* stream) {
    msparse_status st = check_dims(dims, false);
    if (st) return st;
    if (!q || !k || !v || !out || !dout || !lse || !dq || !dk || !dv)
        return fail(MSPARSE_ERR_INVALID, "tensor pointer is NULL");
    if (misaligned({q, k, v, out, out_f32, dout, lse, dq, dk, dv}))
        return fail(MSPARSE_ERR_INVALID, "tensor not 16-byte aligned");
    if ((st = check_index_struct(dims, index, true))) return st;
    if (flags & ~(MSPARSE_BWD_ACCUMULATE_DQ | MSPARSE_BWD_REUSE_QROWS))
        return fail(MSPARSE_ERR_INVALID, "backward flags 0x%x", unsigned(flags));
    const size_t need = msparse_attn_bwd_workspace(dims, index->vcol_cap);
    if (!ws || ws_bytes < need) return fail(MSPARSE_ERR_WORKSPACE, "bwd workspace %zu < %zu bytes", ws_bytes, need);
    if (dims->seq_q == 0 && dims->seq_k == 0) return MSPARSE_OK;
    AttnArgs a{};
    fill_attn(dims, index, &a);
    carve_bwd(dims, index->vcol_cap, static_cast<char*>(ws), &a);
    a.vcol_cap = index->vcol_cap;
    a.o_f32 = out_f32;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = static_cast<const uint16_t*>(out);
    a.dout = static_cast<const uint16_t*>(dout);
    a.lse = const_cast<float*>(lse);
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.dq_accumulate = (flags & MSPARSE_BWD_ACCUMULATE_DQ) != 0;
    a.reuse_qrows = (flags & MSPARSE_BWD_REUSE_QROWS) != 0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return check_hip(launch_attn_bwd(a, s), s, "attn bwd");
}

// ------------------------------------------------------------------ ring workload
msparse_status msparse_ring_work(const msparse_dims* dims, const int32_t* v_idx, int32_t k_v, const int32_t* s_idx,
                                 int32_t k_s, int32_t world, int32_t layout, int64_t* tiles, int64_t* cols, void* ws,
                                 size_t ws_bytes, void* stream) {
    RingInfo ri;
    msparse_status st = check_index_inputs(dims, v_idx, k_v, s_idx, k_s, nullptr, &ri);
    if (st) return st;
    if (!tiles || !cols) return fail(MSPARSE_ERR_INVALID, "workload outputs are NULL");
    if (world < 1 || world > kMaxRingWorld) return fail(MSPARSE_ERR_INVALID, "world %d outside [1, %d]", world, kMaxRingWorld);
    if (layout != MSPARSE_LAYOUT_STRIPED && layout != MSPARSE_LAYOUT_ZIGZAG)
        return fail(MSPARSE_ERR_INVALID, "ring layout %d", layout);
    const int32_t nb = dims->seq_q / kBlock;
    const int32_t unit = layout == MSPARSE_LAYOUT_ZIGZAG ? 2 * world : world;
    if (nb % unit != 0)
        return fail(MSPARSE_ERR_UNSUPPORTED, "%d blocks do not split into %d equal %s shards", nb, world,
                    layout == MSPARSE_LAYOUT_ZIGZAG ? "zigzag" : "striped");
    IndexPlan p = plan_index(dims, k_v, k_s, ri, ws, true);
    if (!ws || ws_bytes < p.bytes)
        return fail(MSPARSE_ERR_WORKSPACE, "index workspace %zu < %zu bytes", ws_bytes, p.bytes);
    p.a.v_idx = v_idx;
    p.a.s_idx = s_idx;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_hip(launch_index_prep(p.a, s), s, "index prep"))) return st;
    return check_hip(launch_ring_work(p.a, world, layout, tiles, cols, s), s, "ring work");
}

// ------------------------------------------------------------------ estimation
size_t msparse_estimate_workspace(const msparse_dims* dims, int32_t last_q, int32_t k_v, int32_t k_s) {
    (void)k_v;
    (void)k_s;
    if (check_dims(dims, true) || last_q < 1) return 0;
    const size_t scores = align_up(size_t(dims->batch) * dims->heads_q * dims->seq_q * sizeof(float));
    return 2 * scores + est_workspace_bytes(dims->batch, dims->heads_q, dims->seq_q, last_q);
}

static msparse_status estimate_impl(const msparse_dims* dims, const void* q, const void* k, int32_t last_q, int32_t k_v,
                                    int32_t k_s, double p_v, double p_s, int32_t* v_idx, int32_t* s_idx, int32_t* v_cnt,
                                    int32_t* s_cnt, float* v_score, float* s_score, void* ws, size_t ws_bytes,
                                    void* stream) {
    msparse_status st = check_dims(dims, true);
    if (st) return st;
    const int32_t N = dims->seq_q;
    if (!q || !k || !v_idx || !s_idx) return fail(MSPARSE_ERR_INVALID, "tensor pointer is NULL");
    if (misaligned({q, k})) return fail(MSPARSE_ERR_INVALID, "tensor not 16-byte aligned");
    if (N < 1) return fail(MSPARSE_ERR_INVALID, "empty sequence");
    if (last_q < 1 || last_q > N) return fail(MSPARSE_ERR_INVALID, "last_q %d outside [1, %d]", last_q, N);
    if (last_q > kBlock) return fail(MSPARSE_ERR_UNSUPPORTED, "last_q %d > 64", last_q);
    if (k_v < 1 || k_v > N || k_s < 1 || k_s > N)
        return fail(MSPARSE_ERR_INVALID, "budgets k_v=%d k_s=%d outside [1, %d]", k_v, k_s, N);
    const size_t need = msparse_estimate_workspace(dims, last_q, k_v, k_s);
    if (!ws || ws_bytes < need) return fail(MSPARSE_ERR_WORKSPACE, "estimate workspace %zu < %zu", ws_bytes, need);
    EstArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.B = dims->batch;
    a.Hq = dims->heads_q;
    a.Hkv = dims->heads_kv;
    a.N = N;
    a.d = dims->head_dim;
    a.L = last_q;
    a.k_v = k_v;
    a.k_s = k_s;
    a.p_v = p_v;
    a.p_s = p_s;
    a.v_cnt = v_cnt;
    a.s_cnt = s_cnt;
    a.scale = resolve_scale(dims);
    a.v_idx = v_idx;
    a.s_idx = s_idx;
    char* base = static_cast<char*>(ws);
    const size_t scores = align_up(size_t(dims->batch) * dims->heads_q * N * sizeof(float));
    a.v_score = v_score ? v_score : reinterpret_cast<float*>(base);
    a.s_score = s_score ? s_score : reinterpret_cast<float*>(base + scores);
    est_carve(a, base + 2 * scores);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return check_hip(launch_estimate(a, s), s, "estimate");
}

msparse_status msparse_estimate(const msparse_dims* dims, const void* q, const void* k, int32_t last_q, int32_t k_v,
                                int32_t k_s, int32_t* v_idx, int32_t* s_idx, float* v_score, float* s_score, void* ws,
                                size_t ws_bytes, void* stream) {
    return estimate_impl(dims, q, k, last_q, k_v, k_s, 0.0, 0.0, v_idx, s_idx, nullptr, nullptr, v_score, s_score, ws,
                         ws_bytes, stream);
}

size_t msparse_estimate_topp_workspace(const msparse_dims* dims, int32_t last_q, int32_t kmax_v, int32_t kmax_s) {
    return msparse_estimate_workspace(dims, last_q, kmax_v, kmax_s);
}

msparse_status msparse_estimate_topp(const msparse_dims* dims, const void* q, const void* k, int32_t last_q, double p_v,
                                     double p_s, int32_t kmax_v, int32_t kmax_s, int32_t* v_idx, int32_t* s_idx,
                                     int32_t* v_cnt, int32_t* s_cnt, float* v_score, float* s_score, void* ws,
                                     size_t ws_bytes, void* stream) {
    if (!(p_v > 0.0 && p_v < 1.0) || !(p_s > 0.0 && p_s < 1.0))
        return fail(MSPARSE_ERR_INVALID, "top-p fractions p_v=%g p_s=%g outside (0, 1)", p_v, p_s);
    if (!v_cnt || !s_cnt) return fail(MSPARSE_ERR_INVALID, "budget output pointer is NULL");
    return estimate_impl(dims, q, k, last_q, kmax_v, kmax_s, p_v, p_s, v_idx, s_idx, v_cnt, s_cnt, v_score, s_score,
                         ws, ws_bytes, stream);
}

}  // extern "C"
