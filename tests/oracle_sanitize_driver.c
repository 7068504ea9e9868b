/*
 * Drives every entry point of the C oracle (oracle/c3_oracle.c) on edge
 * inputs so that a build with -fsanitize=address,undefined checks its memory
 * accesses and integer arithmetic.  Test infrastructure: compiled and run by
 * tests/test_sanitize.py on the CPU only.
 *
 * Every input buffer is its own heap allocation of exactly the bytes the
 * call may read (tensor bytes, evidence rows, bitmaps), so a read past a
 * ragged chunk end or past the last unit is reported by AddressSanitizer.
 * The driver also checks a few results whose values are fixed by the
 * definition (identical replicas agree, one changed byte is attributed to
 * its replica and chunk, caps bound the lists) and prints "ok" at the end.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void c3o_keys(uint32_t *K);
int64_t c3o_num_chunks(const int32_t *dtypes, const int32_t *ndims, const int64_t *shapes, int T,
                       uint64_t chunk_bytes);
int c3o_signature(const uint8_t *const *ptrs, const int32_t *dtypes, const int32_t *ndims,
                  const int64_t *shapes, int T, int R, uint64_t chunk_bytes, uint64_t *sig,
                  uint64_t *n_elems, uint32_t *nan_count, uint32_t *inf_count, double *absmax,
                  double *sum, double *sumsq, uint32_t *tensor_id, uint32_t *chunk_id);
int c3o_tensor_signature(const uint64_t *sig, const uint32_t *tensor_id, int R, int64_t C, int T,
                         uint64_t *out);
int c3o_vote_exact(const uint8_t *evidence, int kind, int64_t replica_stride, int64_t unit_stride,
                   int R, int64_t n_units, uint8_t *status, uint64_t *bitmap, int32_t *majority_idx);
int c3o_vote_bytes(const uint8_t *const *chunk_ptrs, const uint64_t *chunk_len, int R,
                   int64_t n_units, uint8_t *status, uint64_t *bitmap, int32_t *majority_idx);
int c3o_vote_statistical(const uint8_t *evidence, int kind, int64_t replica_stride,
                         int64_t unit_stride, int R, int64_t n_units, double kappa, uint8_t *status,
                         uint64_t *bitmap, int32_t *majority_idx);
int c3o_localize(const uint8_t *status, const uint64_t *bitmap, const int32_t *majority_idx, int R,
                 int64_t n_units, int64_t *out_unit, int32_t *out_replica, int32_t *out_majority,
                 int64_t out_cap, int64_t *undecided, int64_t und_cap, int64_t *counts);
int c3o_confirm(const uint64_t *fp_bitmap, const uint64_t *time_bitmap, int R, int64_t G, int64_t T,
                int W, uint32_t *flags, int32_t *first_div, uint32_t *div_count,
                uint32_t *slow_count, uint32_t *max_window, int32_t *first_window);

#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            exit(1);                                                      \
        }                                                                 \
    } while (0)

static uint64_t rng_state = 0x2545F4914F6CDD1DULL;
static uint64_t rnd(void) { /* xorshift64 */
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return rng_state;
}

static void *xmalloc(size_t n) {
    void *p = malloc(n ? n : 1);
    CHECK(p != NULL);
    return p;
}

static const int ESIZE[4] = {4, 2, 2, 1};

/* Special element patterns per dtype: zeros, sign, subnormal, Inf, NaN. */
static void plant_specials(uint8_t *b, uint64_t nbytes, int dtype) {
    static const uint32_t f32[] = {0u, 0x80000000u, 1u, 0x7F800000u, 0xFF800000u, 0x7FC00000u,
                                   0x7F800001u, 0x007FFFFFu};
    static const uint16_t b16[] = {0u, 0x8000u, 1u, 0x7F80u, 0xFF80u, 0x7FC0u, 0x7F81u, 0x007Fu};
    static const uint16_t h16[] = {0u, 0x8000u, 1u, 0x7C00u, 0xFC00u, 0x7E00u, 0x7C01u, 0x03FFu};
    uint64_t n = nbytes / (uint64_t)ESIZE[dtype], i;
    for (i = 0; i < 8 && 5 * i < n; i++) {
        if (dtype == 0) memcpy(b + 4 * (5 * i), &f32[i], 4);
        if (dtype == 1) memcpy(b + 2 * (5 * i), &b16[i], 2);
        if (dtype == 2) memcpy(b + 2 * (5 * i), &h16[i], 2);
    }
}

static void signature_cases(void) {
    static const int64_t sizes[] = {0, 1, 3, 7, 8, 9, 255, 256, 257, 511, 4097};
    const int T = (int)(sizeof(sizes) / sizeof(sizes[0])), R = 3;
    static const uint64_t chunks[] = {1024, 3072, 8192};
    int dtype, ci;
    for (dtype = 0; dtype < 4; dtype++) {
        for (ci = 0; ci < 3; ci++) {
            const uint64_t cb = chunks[ci];
            int32_t dtypes[16], ndims[16];
            int64_t shapes[16 * 8];
            uint8_t *ptrs[3 * 16];
            int64_t C, i;
            int r, t;
            memset(shapes, 0, sizeof(shapes));
            for (t = 0; t < T; t++) {
                dtypes[t] = dtype;
                ndims[t] = 1;
                shapes[8 * t] = sizes[t];
            }
            C = c3o_num_chunks(dtypes, ndims, shapes, T, cb);
            CHECK(C >= T);
            for (t = 0; t < T; t++) {
                uint64_t nb = (uint64_t)sizes[t] * (uint64_t)ESIZE[dtype];
                uint8_t *b0 = (uint8_t *)xmalloc(nb);
                uint64_t k;
                for (k = 0; k < nb; k++) b0[k] = (uint8_t)rnd();
                plant_specials(b0, nb, dtype);
                for (r = 0; r < R; r++) {
                    ptrs[r * T + t] = (uint8_t *)xmalloc(nb);
                    if (nb) memcpy(ptrs[r * T + t], b0, nb);
                }
                free(b0);
            }
            /* one changed byte in the last byte of tensor 8 on replica 1 */
            {
                uint64_t nb8 = (uint64_t)sizes[8] * (uint64_t)ESIZE[dtype];
                ptrs[1 * T + 8][nb8 - 1] ^= 0x01;
            }
            {
                uint64_t *sig = (uint64_t *)xmalloc(8 * (size_t)(R * C));
                uint64_t *ne = (uint64_t *)xmalloc(8 * (size_t)(R * C));
                uint32_t *nan = (uint32_t *)xmalloc(4 * (size_t)(R * C));
                uint32_t *inf = (uint32_t *)xmalloc(4 * (size_t)(R * C));
                double *amax = (double *)xmalloc(8 * (size_t)(R * C));
                double *sum = (double *)xmalloc(8 * (size_t)(R * C));
                double *sq = (double *)xmalloc(8 * (size_t)(R * C));
                uint32_t *tid = (uint32_t *)xmalloc(4 * (size_t)(R * C));
                uint32_t *cid = (uint32_t *)xmalloc(4 * (size_t)(R * C));
                uint64_t *tsig = (uint64_t *)xmalloc(8 * (size_t)(R * T));
                uint8_t *st = (uint8_t *)xmalloc((size_t)C);
                uint64_t *bm = (uint64_t *)xmalloc(8 * (size_t)C);
                int32_t *mj = (int32_t *)xmalloc(4 * (size_t)C);
                int64_t n_att = 0;
                CHECK(c3o_signature((const uint8_t *const *)ptrs, dtypes, ndims, shapes, T, R, cb,
                                    sig, ne, nan, inf, amax, sum, sq, tid, cid) == 0);
                CHECK(c3o_tensor_signature(sig, tid, R, C, T, tsig) == 0);
                /* signature vote over the [R][C] table */
                CHECK(c3o_vote_exact((const uint8_t *)sig, 0, 8 * C, 8, R, C, st, bm, mj) == 0);
                for (i = 0; i < C; i++) {
                    if (st[i] == 1) {
                        n_att++;
                        CHECK(bm[i] == 2u && tid[i] == 8u);
                    } else {
                        CHECK(st[i] == 0);
                    }
                }
                CHECK(n_att == 1);
                for (i = 0; i < C; i++)
                    CHECK(isfinite(sum[i]) && isfinite(sq[i]) && isfinite(amax[i]));
                free(sig); free(ne); free(nan); free(inf); free(amax); free(sum); free(sq);
                free(tid); free(cid); free(tsig); free(st); free(bm); free(mj);
            }
            for (r = 0; r < R * T; r++) free(ptrs[r]);
        }
    }
}

static void vote_cases(void) {
    int R;
    for (R = 2; R <= 64; R++) {
        const int64_t U = 97;
        uint64_t *ev = (uint64_t *)xmalloc(8 * (size_t)(U * R));
        uint32_t *ev32 = (uint32_t *)xmalloc(4 * (size_t)(U * R));
        double *tf64 = (double *)xmalloc(8 * (size_t)(U * R));
        float *tf32 = (float *)xmalloc(4 * (size_t)(U * R));
        uint8_t *st = (uint8_t *)xmalloc((size_t)U);
        uint64_t *bm = (uint64_t *)xmalloc(8 * (size_t)U);
        int32_t *mj = (int32_t *)xmalloc(4 * (size_t)U);
        const uint8_t **cp = (const uint8_t **)xmalloc(sizeof(uint8_t *) * (size_t)(U * R));
        uint64_t *cl = (uint64_t *)xmalloc(8 * (size_t)U);
        int64_t u, cnt[3];
        int r;
        for (u = 0; u < U; u++) {
            for (r = 0; r < R; r++) {
                const uint64_t label = rnd() % 3 == 0 ? rnd() % 3 : 0;
                ev[u * R + r] = label;
                ev32[u * R + r] = (uint32_t)label;
                tf64[u * R + r] = 1.0 + 0.01 * (double)(rnd() % 7);
                if (rnd() % 29 == 0) tf64[u * R + r] = NAN;
                if (rnd() % 31 == 0) tf64[u * R + r] = INFINITY;
                if (u % 11 == 0) tf64[u * R + r] = 2.0; /* all equal: every scale is 0 */
                tf32[u * R + r] = (float)tf64[u * R + r];
                cp[r * U + u] = (const uint8_t *)&ev[u * R + r];
            }
            cl[u] = 8;
        }
        /* a singleton group is refused before anything is read (Sec. 4) */
        CHECK(c3o_vote_exact((const uint8_t *)ev, 0, 8, 8 * R, 1, U, st, bm, mj) == -1);
        CHECK(c3o_vote_exact((const uint8_t *)ev, 0, 8, 8 * R, R, U, st, bm, mj) == 0);
        CHECK(c3o_vote_exact((const uint8_t *)ev32, 1, 4, 4 * R, R, U, st, bm, mj) == 0);
        CHECK(c3o_vote_bytes((const uint8_t *const *)cp, cl, R, U, st, bm, mj) == 0);
        CHECK(c3o_vote_statistical((const uint8_t *)tf32, 2, 4, 4 * R, R, U, 3.5 / 0.6745, st,
                                   bm, mj) == 0);
        CHECK(c3o_vote_statistical((const uint8_t *)tf64, 3, 8, 8 * R, R, U, 3.5 / 0.6745, st,
                                   bm, mj) == 0);
        for (u = 0; u < U; u++) CHECK(st[u] <= 2 && (R == 64 || (bm[u] >> R) == 0));
        {
            /* lists with caps below, at and above the totals */
            int64_t caps[3] = {0, 3, 64 * U}, c;
            for (c = 0; c < 3; c++) {
                int64_t cap = caps[c];
                int64_t *ou = (int64_t *)xmalloc(8 * (size_t)cap);
                int32_t *orr = (int32_t *)xmalloc(4 * (size_t)cap);
                int32_t *om = (int32_t *)xmalloc(4 * (size_t)cap);
                int64_t *und = (int64_t *)xmalloc(8 * (size_t)cap);
                CHECK(c3o_localize(st, bm, mj, R, U, ou, orr, om, cap, und, cap, cnt) == 0);
                CHECK(cnt[0] >= 0 && cnt[1] >= 0 && cnt[2] >= 0 && cnt[1] <= U);
                free(ou); free(orr); free(om); free(und);
            }
        }
        free(ev); free(ev32); free(tf64); free(tf32); free(st); free(bm); free(mj);
        free(cp); free(cl);
    }
}

static void confirm_cases(void) {
    static const int64_t Ts[] = {0, 1, 2, 31, 32, 33, 64, 65, 130};
    static const int Ws[] = {1, 2, 7, 16, 64, 80, 200};
    size_t a, b;
    for (a = 0; a < sizeof(Ts) / sizeof(Ts[0]); a++) {
        for (b = 0; b < sizeof(Ws) / sizeof(Ws[0]); b++) {
            const int64_t T = Ts[a], G = 5;
            const int R = 13, W = Ws[b];
            uint64_t *fb = (uint64_t *)xmalloc(8 * (size_t)(T * G));
            uint64_t *tb = (uint64_t *)xmalloc(8 * (size_t)(T * G));
            uint32_t *fl = (uint32_t *)xmalloc(4 * (size_t)(R * G));
            int32_t *fd = (int32_t *)xmalloc(4 * (size_t)(R * G));
            uint32_t *dc = (uint32_t *)xmalloc(4 * (size_t)(R * G));
            uint32_t *sc = (uint32_t *)xmalloc(4 * (size_t)(R * G));
            uint32_t *mw = (uint32_t *)xmalloc(4 * (size_t)(R * G));
            int32_t *fw = (int32_t *)xmalloc(4 * (size_t)(R * G));
            int64_t i;
            for (i = 0; i < T * G; i++) {
                fb[i] = rnd() % 5 == 0 ? (rnd() & ((1ULL << R) - 1)) : 0;
                tb[i] = rnd() & ((1ULL << R) - 1);
            }
            CHECK(c3o_confirm(fb, tb, R, G, T, W, fl, fd, dc, sc, mw, fw) == 0);
            for (i = 0; i < R * G; i++) CHECK(sc[i] <= (uint32_t)T && dc[i] <= (uint32_t)T);
            free(fb); free(tb); free(fl); free(fd); free(dc); free(sc); free(mw); free(fw);
        }
    }
}

int main(void) {
    uint32_t K[258];
    c3o_keys(K);
    signature_cases();
    vote_cases();
    confirm_cases();
    printf("ok\n");
    return 0;
}
