/* A plain C caller of the library's C ABI (no Python, no torch): reads a
 * workload from a binary file, runs estimate -> index count -> index build ->
 * forward -> backward on one GPU, and writes the results to a binary file.
 *
 * usage: abi_roundtrip <in.bin> <out.bin>
 * in.bin  int32 [8] = B, N, Hq, Hkv, d, last_q, k_v, k_s, then
 *         q bf16 [B,Hq,N,d], k, v bf16 [B,Hkv,N,d], dO bf16 [B,Hq,N,d],
 *         v_idx int32 [B,Hq,k_v], s_idx int32 [B,Hq,k_s]: the sets the index
 *         is built from (the estimate's own sets are written out beside).
 * out.bin est_v int32 [B,Hq,k_v], est_s int32 [B,Hq,k_s], out bf16 [B,Hq,N,d],
 *         lse fp32 [B,Hq,N], dq fp32 [B,Hq,N,d], dk, dv fp32 [B,Hkv,N,d].
 * Exit status 0 on success; a failing call prints its status and message. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "msparse.h"

static int fail_st(const char* what, msparse_status st) {
    fprintf(stderr, "%s: %s (%s)\n", what, msparse_strerror(st), msparse_last_error());
    return 1;
}

static void* dev_alloc(size_t bytes) {
    void* p = NULL;
    if (hipMalloc(&p, bytes ? bytes : 16) != hipSuccess) {
        fprintf(stderr, "hipMalloc of %zu bytes failed\n", bytes);
        exit(2);
    }
    return p;
}

static void* read_block(FILE* f, size_t bytes) {
    void* h = malloc(bytes ? bytes : 1);
    if (!h || fread(h, 1, bytes, f) != bytes) {
        fprintf(stderr, "short input\n");
        exit(2);
    }
    return h;
}

static void* to_dev(const void* h, size_t bytes) {
    void* d = dev_alloc(bytes);
    hipMemcpy(d, h, bytes, hipMemcpyHostToDevice);
    return d;
}

static void write_dev(FILE* f, const void* d, size_t bytes) {
    void* h = malloc(bytes ? bytes : 1);
    hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost);
    fwrite(h, 1, bytes, f);
    free(h);
}

int main(int argc, char** argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s in.bin out.bin\n", argv[0]);
        return 2;
    }
    FILE* fi = fopen(argv[1], "rb");
    if (!fi) return 2;
    int32_t hd[8];
    if (fread(hd, sizeof(int32_t), 8, fi) != 8) return 2;
    const int32_t B = hd[0], N = hd[1], Hq = hd[2], Hkv = hd[3], d = hd[4], last_q = hd[5], k_v = hd[6], k_s = hd[7];
    const size_t nq = (size_t)B * Hq * N * d, nkv = (size_t)B * Hkv * N * d, rows = (size_t)B * Hq * N;
    void* q = to_dev(read_block(fi, nq * 2), nq * 2);
    void* k = to_dev(read_block(fi, nkv * 2), nkv * 2);
    void* v = to_dev(read_block(fi, nkv * 2), nkv * 2);
    void* dout = to_dev(read_block(fi, nq * 2), nq * 2);
    int32_t* vi = (int32_t*)to_dev(read_block(fi, (size_t)B * Hq * k_v * 4), (size_t)B * Hq * k_v * 4);
    int32_t* si = (int32_t*)to_dev(read_block(fi, (size_t)B * Hq * k_s * 4), (size_t)B * Hq * k_s * 4);
    fclose(fi);

    msparse_dims dims;
    memset(&dims, 0, sizeof(dims));
    dims.batch = B;
    dims.seq_q = N;
    dims.seq_k = N;
    dims.heads_q = Hq;
    dims.heads_kv = Hkv;
    dims.head_dim = d;
    dims.block = 64;
    dims.causal = 1;
    dims.scale = 0.f;
    msparse_status st;

    /* estimate (its sets are written out; the index below uses the given ones) */
    int32_t* ev = (int32_t*)dev_alloc((size_t)B * Hq * k_v * 4);
    int32_t* es = (int32_t*)dev_alloc((size_t)B * Hq * k_s * 4);
    size_t ews = msparse_estimate_workspace(&dims, last_q, k_v, k_s);
    void* ew = dev_alloc(ews);
    if ((st = msparse_estimate(&dims, q, k, last_q, k_v, k_s, ev, es, NULL, NULL, ew, ews, NULL)))
        return fail_st("estimate", st);

    /* index: exact counts, then the build */
    size_t iws = msparse_index_workspace(&dims, k_v, k_s, NULL);
    void* iw = dev_alloc(iws);
    int64_t nblk = 0, ncol = 0, nvcol = 0;
    if ((st = msparse_index_count(&dims, vi, k_v, si, k_s, NULL, &nblk, &ncol, &nvcol, iw, iws, NULL)))
        return fail_st("index count", st);
    const int64_t nqb = N / 64, bh = (int64_t)B * Hq;
    msparse_index idx;
    memset(&idx, 0, sizeof(idx));
    idx.blk_ptr = (int64_t*)dev_alloc((size_t)(bh * nqb + 1) * 8);
    idx.blk_idx = (int32_t*)dev_alloc((size_t)nblk * 4);
    idx.blk_cap = nblk;
    idx.col_ptr = (int64_t*)dev_alloc((size_t)(bh * nqb + 1) * 8);
    idx.col_idx = (int32_t*)dev_alloc((size_t)ncol * 4);
    idx.col_cap = ncol;
    idx.kblk_ptr = (int64_t*)dev_alloc((size_t)(bh * nqb + 1) * 8);
    idx.kblk_idx = (int32_t*)dev_alloc((size_t)nblk * 4);
    idx.vcol_ptr = (int64_t*)dev_alloc((size_t)(bh + 1) * 8);
    idx.vcol_idx = (int32_t*)dev_alloc((size_t)nvcol * 4);
    idx.vcol_cap = nvcol;
    idx.diag_bits = (uint32_t*)dev_alloc((size_t)bh * ((nqb + 31) / 32) * 4);
    idx.q_blk_global = (int32_t*)dev_alloc((size_t)nqb * 4);
    idx.k_blk_global = (int32_t*)dev_alloc((size_t)nqb * 4);
    idx.overflow = (int32_t*)dev_alloc(4);
    idx.world = 1;
    if ((st = msparse_build_index(&dims, vi, k_v, si, k_s, NULL, &idx, iw, iws, NULL)))
        return fail_st("index build", st);

    /* forward and backward */
    void* out = dev_alloc(nq * 2);
    float* lse = (float*)dev_alloc(rows * 4);
    float* out32 = (float*)dev_alloc(nq * 4);
    size_t fws = msparse_attn_fwd_workspace(&dims);
    void* fw = dev_alloc(fws);
    if ((st = msparse_attn_fwd(&dims, q, k, v, &idx, out, lse, out32, fw, fws, NULL))) return fail_st("fwd", st);
    float* dq = (float*)dev_alloc(nq * 4);
    float* dk = (float*)dev_alloc(nkv * 4);
    float* dv = (float*)dev_alloc(nkv * 4);
    size_t bws = msparse_attn_bwd_workspace(&dims, idx.vcol_cap);
    void* bw = dev_alloc(bws);
    if ((st = msparse_attn_bwd(&dims, q, k, v, out, out32, dout, lse, &idx, dq, dk, dv, 0, bw, bws, NULL)))
        return fail_st("bwd", st);
    if (hipDeviceSynchronize() != hipSuccess) {
        fprintf(stderr, "device error\n");
        return 1;
    }
    int32_t ovf = 0;
    hipMemcpy(&ovf, idx.overflow, 4, hipMemcpyDeviceToHost);
    if (ovf) {
        fprintf(stderr, "index overflowed with exact capacities\n");
        return 1;
    }

    FILE* fo = fopen(argv[2], "wb");
    if (!fo) return 2;
    write_dev(fo, ev, (size_t)B * Hq * k_v * 4);
    write_dev(fo, es, (size_t)B * Hq * k_s * 4);
    write_dev(fo, out, nq * 2);
    write_dev(fo, lse, rows * 4);
    write_dev(fo, dq, nq * 4);
    write_dev(fo, dk, nkv * 4);
    write_dev(fo, dv, nkv * 4);
    fclose(fo);
    printf("abi_roundtrip ok: %lld block entries, %lld column entries\n", (long long)nblk, (long long)ncol);
    return 0;
}
