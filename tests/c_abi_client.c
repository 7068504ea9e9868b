/*
 * A plain C client of libc3.so: no Python, no torch.  It allocates device
 * memory with the HIP runtime, signs R replicas of one ragged fp32 tensor,
 * votes per chunk and localizes, then checks what the definition fixes:
 *   - identical replicas: every chunk agrees, empty lists;
 *   - one flipped bit in replica 2: exactly (replica 2, the element's chunk)
 *     is attributed, majority replica 0, no undecided chunk;
 *   - the outlier's summary is the records' (NaN count after an exponent
 *     flip that makes a NaN, absmax of the majority);
 *   - argument errors come back as codes with nothing launched;
 *   - a 130-replica group (C3_BITMAP_WORDS(130) = 3 words per unit): the
 *     outliers planted in replicas 1, 64 and 129 land in the right words and
 *     list entries, a replica-0 fault is attributed with majority replica 1.
 * Built by the package build next to libc3.so; run by tests/test_gpu_c_abi.py.
 * Prints "ok" and exits 0 on success.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "c3.h"

#define HIP_OK(x)                                                                    \
    do {                                                                             \
        hipError_t e_ = (x);                                                         \
        if (e_ != hipSuccess) {                                                      \
            fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, hipGetErrorString(e_)); \
            exit(2);                                                                 \
        }                                                                            \
    } while (0)
#define CHECK(c)                                                        \
    do {                                                                \
        if (!(c)) {                                                     \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
            exit(1);                                                    \
        }                                                               \
    } while (0)

enum { R = 3, N = 1000003 };
static const uint64_t CHUNK = 65536;

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (uint32_t)(rng >> 11);
}

struct run {
    int64_t counts[3];
    c3_outlier_t outliers[8];
    int64_t undecided[8];
    uint8_t status[64];
};

static void run_path(float *const *dev, const c3_tensor_meta_t *meta, int64_t C, void *ws,
                     size_t ws_bytes, c3_chunk_record_t *rec, uint8_t *st, uint64_t *bm, int32_t *mj,
                     c3_outlier_t *outl, int64_t *und, int64_t *cnt, void *lws, size_t lws_bytes,
                     hipStream_t s, struct run *out) {
    const void *ptrs[R];
    int r;
    for (r = 0; r < R; ++r) ptrs[r] = dev[r];
    CHECK(c3_signature(ptrs, meta, 1, R, CHUNK, rec, ws, ws_bytes, (c3_stream_t)s) == C3_OK);
    CHECK(c3_consensus(rec, C3_EV_U64, C * (int64_t)sizeof(c3_chunk_record_t),
                       (int64_t)sizeof(c3_chunk_record_t), R, C, C3_EXACT, C3_KAPPA_DEFAULT, st, bm,
                       mj, (c3_stream_t)s) == C3_OK);
    CHECK(c3_localize(st, bm, mj, rec, R, C, outl, 8, und, 8, cnt, lws, lws_bytes,
                      (c3_stream_t)s) == C3_OK);
    HIP_OK(hipStreamSynchronize(s));
    HIP_OK(hipMemcpy(out->counts, cnt, sizeof(out->counts), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(out->outliers, outl, sizeof(out->outliers), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(out->undecided, und, sizeof(out->undecided), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(out->status, st, (size_t)C, hipMemcpyDeviceToHost));
}

int main(void) {
    c3_tensor_meta_t meta;
    memset(&meta, 0, sizeof(meta));
    meta.dtype = C3_F32;
    meta.ndim = 1;
    meta.shape[0] = N;
    const int64_t C = c3_num_chunks(&meta, 1, CHUNK);
    CHECK(C == (int64_t)((4ull * N + CHUNK - 1) / CHUNK) && C <= 64);
    const size_t ws_bytes = c3_signature_workspace_size(&meta, 1, R, CHUNK);
    const size_t lws_bytes = c3_localize_workspace_size(C);
    CHECK(ws_bytes > 0 && lws_bytes > 0);
    CHECK(c3_abi_version() == C3_ABI_VERSION);
    CHECK(strcmp(c3_status_string(C3_E_ALIGN), "misaligned pointer or stride") == 0);

    float *host = (float *)malloc(4 * (size_t)N);
    CHECK(host != NULL);
    for (int i = 0; i < N; ++i) host[i] = (float)((int)(next_u32() % 20001) - 10000) * 1e-4f;

    hipStream_t s;
    HIP_OK(hipStreamCreate(&s));
    float *dev[R];
    void *ws, *lws;
    c3_chunk_record_t *rec;
    uint8_t *st;
    uint64_t *bm;
    int32_t *mj;
    c3_outlier_t *outl;
    int64_t *und, *cnt;
    for (int r = 0; r < R; ++r) {
        HIP_OK(hipMalloc((void **)&dev[r], 4 * (size_t)N));
        HIP_OK(hipMemcpy(dev[r], host, 4 * (size_t)N, hipMemcpyHostToDevice));
    }
    HIP_OK(hipMalloc(&ws, ws_bytes));
    HIP_OK(hipMalloc(&lws, lws_bytes));
    HIP_OK(hipMalloc((void **)&rec, sizeof(c3_chunk_record_t) * (size_t)(R * C)));
    HIP_OK(hipMalloc((void **)&st, (size_t)C));
    HIP_OK(hipMalloc((void **)&bm, 8 * (size_t)C));
    HIP_OK(hipMalloc((void **)&mj, 4 * (size_t)C));
    HIP_OK(hipMalloc((void **)&outl, sizeof(c3_outlier_t) * 8));
    HIP_OK(hipMalloc((void **)&und, 8 * 8));
    HIP_OK(hipMalloc((void **)&cnt, 8 * 3));

    /* identical replicas */
    struct run a;
    run_path(dev, &meta, C, ws, ws_bytes, rec, st, bm, mj, outl, und, cnt, lws, lws_bytes, s, &a);
    CHECK(a.counts[0] == 0 && a.counts[1] == 0 && a.counts[2] == 0);
    for (int64_t c = 0; c < C; ++c) CHECK(a.status[c] == C3_AGREE);

    /* replica 2: exponent bits of one element set, which makes it a NaN */
    const int64_t elem = 777777;
    uint32_t bits;
    memcpy(&bits, &host[elem], 4);
    bits |= 0x7FC00000u;
    HIP_OK(hipMemcpy((char *)dev[2] + 4 * elem, &bits, 4, hipMemcpyHostToDevice));
    struct run b;
    run_path(dev, &meta, C, ws, ws_bytes, rec, st, bm, mj, outl, und, cnt, lws, lws_bytes, s, &b);
    CHECK(b.counts[0] == 1 && b.counts[1] == 0 && b.counts[2] == 1);
    CHECK(b.outliers[0].chunk == (int64_t)((uint64_t)elem * 4 / CHUNK));
    CHECK(b.outliers[0].replica == 2 && b.outliers[0].majority_replica == 0);
    CHECK(b.outliers[0].nan_count[0] == 1 && b.outliers[0].nan_count[1] == 0);
    CHECK(b.outliers[0].inf_count[0] == 0 && b.outliers[0].inf_count[1] == 0);
    CHECK(b.outliers[0].absmax[1] > 0.0 && b.outliers[0].absmax[1] <= 1.0);
    CHECK(isfinite(b.outliers[0].sum[0]) && isfinite(b.outliers[0].sum[1]));
    for (int64_t c = 0; c < C; ++c)
        CHECK(b.status[c] == (c == b.outliers[0].chunk ? C3_ATTRIBUTED : C3_AGREE));

    /* a wide peer group: U units x 130 replicas of u64 evidence, unit-major */
    {
        enum { RW = 130, UW = 1000 };
        const int W = C3_BITMAP_WORDS(RW);
        uint64_t *hev = (uint64_t *)malloc(sizeof(uint64_t) * RW * UW);
        uint64_t *dev_ev, *dbm, hbm[3];
        uint8_t *dst, hst[UW];
        int32_t *dmj, hmj[UW];
        CHECK(W == 3 && hev != NULL);
        for (int u = 0; u < UW; ++u)
            for (int r = 0; r < RW; ++r) hev[(size_t)u * RW + r] = 0x1234567890ull * (uint64_t)(u + 1);
        hev[(size_t)10 * RW + 1] ^= 1;   /* unit 10: replica 1 (word 0) */
        hev[(size_t)10 * RW + 64] ^= 2;  /* unit 10: replica 64 (word 1) */
        hev[(size_t)500 * RW + 129] ^= 4; /* unit 500: replica 129 (word 2) */
        hev[(size_t)777 * RW + 0] ^= 8;  /* unit 777: replica 0 is the outlier */
        HIP_OK(hipMalloc((void **)&dev_ev, sizeof(uint64_t) * RW * UW));
        HIP_OK(hipMalloc((void **)&dbm, sizeof(uint64_t) * W * UW));
        HIP_OK(hipMalloc((void **)&dst, UW));
        HIP_OK(hipMalloc((void **)&dmj, 4 * UW));
        HIP_OK(hipMemcpy(dev_ev, hev, sizeof(uint64_t) * RW * UW, hipMemcpyHostToDevice));
        CHECK(c3_consensus(dev_ev, C3_EV_U64, 8, 8 * RW, RW, UW, C3_EXACT, C3_KAPPA_DEFAULT, dst,
                           dbm, dmj, (c3_stream_t)s) == C3_OK);
        {
            const size_t lw = c3_localize_workspace_size(UW);
            void *dlws;
            c3_outlier_t o[8];
            int64_t cw[3];
            HIP_OK(hipMalloc(&dlws, lw));
            CHECK(c3_localize(dst, dbm, dmj, NULL, RW, UW, outl, 8, und, 8, cnt, dlws, lw,
                              (c3_stream_t)s) == C3_OK);
            HIP_OK(hipStreamSynchronize(s));
            HIP_OK(hipMemcpy(cw, cnt, sizeof(cw), hipMemcpyDeviceToHost));
            HIP_OK(hipMemcpy(o, outl, sizeof(o), hipMemcpyDeviceToHost));
            CHECK(cw[0] == 4 && cw[1] == 0 && cw[2] == 3);
            CHECK(o[0].chunk == 10 && o[0].replica == 1 && o[0].majority_replica == 0);
            CHECK(o[1].chunk == 10 && o[1].replica == 64);
            CHECK(o[2].chunk == 500 && o[2].replica == 129);
            CHECK(o[3].chunk == 777 && o[3].replica == 0 && o[3].majority_replica == 1);
            HIP_OK(hipFree(dlws));
        }
        HIP_OK(hipMemcpy(hst, dst, UW, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(hmj, dmj, 4 * UW, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(hbm, dbm + (size_t)10 * W, sizeof(hbm), hipMemcpyDeviceToHost));
        CHECK(hbm[0] == 2ull && hbm[1] == 1ull && hbm[2] == 0ull);
        HIP_OK(hipMemcpy(hbm, dbm + (size_t)500 * W, sizeof(hbm), hipMemcpyDeviceToHost));
        CHECK(hbm[0] == 0ull && hbm[1] == 0ull && hbm[2] == 2ull);
        for (int u = 0; u < UW; ++u) {
            const int bad = u == 10 || u == 500 || u == 777;
            CHECK(hst[u] == (bad ? C3_ATTRIBUTED : C3_AGREE));
            CHECK(hmj[u] == (u == 777 ? 1 : 0));
        }
        CHECK(c3_consensus(dev_ev, C3_EV_U64, 8, 8 * RW, C3_MAX_PEERS + 1, UW, C3_EXACT,
                           C3_KAPPA_DEFAULT, dst, dbm, dmj, (c3_stream_t)s) == C3_E_INVAL);
        HIP_OK(hipFree(dev_ev));
        HIP_OK(hipFree(dbm));
        HIP_OK(hipFree(dst));
        HIP_OK(hipFree(dmj));
        free(hev);
    }

    /* argument errors return codes and launch nothing */
    {
        const void *ptrs[R] = {dev[0], dev[1], (const char *)dev[2] + 4};
        CHECK(c3_signature(ptrs, &meta, 1, R, CHUNK, rec, ws, ws_bytes, (c3_stream_t)s) ==
              C3_E_ALIGN);
        CHECK(c3_signature(ptrs, &meta, 1, 0, CHUNK, rec, ws, ws_bytes, (c3_stream_t)s) ==
              C3_E_INVAL);
        CHECK(c3_signature(ptrs, &meta, 1, R, 1000, rec, ws, ws_bytes, (c3_stream_t)s) ==
              C3_E_INVAL);
        /* a group of one replica provides no comparison (Sec. 4): no vote */
        CHECK(c3_consensus(&rec[0].sig, C3_EV_U64, C * (int64_t)sizeof(c3_chunk_record_t),
                           (int64_t)sizeof(c3_chunk_record_t), 1, C, C3_EXACT,
                           C3_KAPPA_DEFAULT, st, bm, mj, (c3_stream_t)s) == C3_E_INVAL);
        CHECK(c3_signature(ptrs, &meta, 1, R, CHUNK, rec, ws, 16, (c3_stream_t)s) ==
              C3_E_WORKSPACE);
    }
    HIP_OK(hipStreamSynchronize(s));

    for (int r = 0; r < R; ++r) HIP_OK(hipFree(dev[r]));
    HIP_OK(hipFree(ws));
    HIP_OK(hipFree(lws));
    HIP_OK(hipFree(rec));
    HIP_OK(hipFree(st));
    HIP_OK(hipFree(bm));
    HIP_OK(hipFree(mj));
    HIP_OK(hipFree(outl));
    HIP_OK(hipFree(und));
    HIP_OK(hipFree(cnt));
    HIP_OK(hipStreamDestroy(s));
    free(host);
    printf("ok\n");
    return 0;
}
