/*
 * C3 oracle: plain, slow, single-threaded CPU implementation of the
 * data-parallel hot path of Consensus Collective Communication (C3).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or constant
 * generator with the HIP implementation; every value here is derived from
 * the paper or from the published definition of a textbook routine:
 *
 *   - SplitMix64 (Steele, Lea, Flood, OOPSLA 2014)        -> key table
 *   - NH hash (Black et al., "UMAC", CRYPTO 1999)          -> chunk fold
 *   - MurmurHash3 fmix64 finalizer (Appleby, public domain) -> finalize
 *   - Neumaier compensated summation (Neumaier 1974)      -> sum, sumsq
 *   - Hyndman-Fan type-7 quantiles                         -> IQR fallback
 *   - Iglewicz-Hoaglin modified z-score (3.5 / 0.6745)     -> kappa default
 *
 * Paper passages followed (section / algorithm / equation):
 *   - Sec. 5.1, Algorithm 1: result R = (s, B, E); statuses Agree,
 *     Attributed, Inconclusive; N-bit outlier bitmap.
 *   - Sec. 5.2: comparable evidence e_i = H_w(dtype, shape, bytes), a
 *     deterministic position-sensitive w-bit hash; w = 64.  The paper gives
 *     no construction for H_w; the construction below (C3SIG-1) is this
 *     implementation's reading, applied per chunk of each tensor.
 *   - Sec. 5.3: exact consensus (most frequent value, strict majority).
 *   - Sec. 5.4: statistical consensus (median, MAD -> IQR -> scaled range,
 *     kappa multiplier).
 *   - Sec. 4 (peer-group size): a two-member disagreement is group-scoped,
 *     i.e. no strict majority, i.e. Inconclusive; a group of one peer has
 *     nothing to compare with, so every vote, localization and confirmation
 *     below rejects R = 1 (returns -1) instead of certifying agreement.
 *   - Sec. 10 (protocol): stragglers are confirmed over repeated rounds.
 *
 * Parity status per function:
 *   c3o_splitmix64_next     pinned (published test vectors)
 *   c3o_fmix64              pinned (bijectivity via an independently derived
 *                           inverse; avalanche); exact constants are the
 *                           published MurmurHash3 ones
 *   c3o_chunk_signature     hash bits: the paper fixes no construction, so the
 *                           bits are C3SIG-1's definition.  Pinned by a
 *                           restatement of that definition in Python integers
 *                           (keys, NH fold and the whole fmix64 chain) and by
 *                           frozen known-answer vectors; indirectly also by
 *                           byte-equality vote == signature vote and
 *                           exhaustive single-bit-flip detection.
 *                           stats: pinned against numpy / math.fsum.
 *   c3o_tensor_signature    pinned by the same restatement and vectors; its
 *                           vote equals the byte-equality vote over whole
 *                           tensors
 *   c3o_vote_exact          pinned (brute force over all label vectors, paper
 *                           cases, Boyer-Moore MJRTY; groups of 65-256 by
 *                           rows whose vote is fixed by construction)
 *   c3o_vote_bytes          the definition itself (byte equality)
 *   c3o_vote_statistical    pinned (numpy median / percentile, closed forms,
 *                           up to 256 replicas)
 *   c3o_localize            pinned (brute-force enumeration of set bits over
 *                           every bitmap word)
 *   c3o_confirm             pinned (brute-force window enumeration)
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -shared -fPIC (no FMA
 * contraction, so every fp64 operation below rounds exactly once).
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#include <math.h>

/* ------------------------------------------------------------------ */
/* Codes.  Values are part of the C ABI of the method (the same numbers */
/* are written independently in the product header).                   */
/* ------------------------------------------------------------------ */
enum { O_F32 = 0, O_BF16 = 1, O_F16 = 2, O_RAW = 3 };
enum { O_AGREE = 0, O_ATTRIBUTED = 1, O_INCONCLUSIVE = 2 };
enum { O_EV_U64 = 0, O_EV_U32 = 1, O_EV_F32 = 2, O_EV_F64 = 3 };

/* ------------------------------------------------------------------ */
/* Peer groups of up to O_MAX_R replicas (the data-parallel peer        */
/* degrees the paper tabulates reach 192, Table 2).  The outlier bitmap */
/* B of a unit is N bits (Sec. 5.1): ceil(R / 64) 64-bit words, bit b   */
/* of word w naming replica 64 w + b.  For R <= 64 that is one word.    */
/* ------------------------------------------------------------------ */
enum { O_MAX_R = 256 };

static int bm_words(int R)
{
    return (R + 63) / 64;
}

static void bm_clear(uint64_t *B, int R)
{
    int w;
    for (w = 0; w < bm_words(R); w++) B[w] = 0;
}

static void bm_set(uint64_t *B, int r)
{
    B[r / 64] |= 1ULL << (r % 64);
}

static int bm_test(const uint64_t *B, int r)
{
    return (int)((B[r / 64] >> (r % 64)) & 1ULL);
}

static int bm_any(const uint64_t *B, int R)
{
    int w;
    for (w = 0; w < bm_words(R); w++)
        if (B[w]) return 1;
    return 0;
}

/* ------------------------------------------------------------------ */
/* SplitMix64 (Steele, Lea, Flood 2014): state advances by the golden   */
/* gamma; output is the mixed state.                                    */
/* ------------------------------------------------------------------ */
uint64_t c3o_splitmix64_next(uint64_t *state)
{
    uint64_t z;
    *state += 0x9E3779B97F4A7C15ULL;
    z = *state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* MurmurHash3 64-bit finalizer (Appleby). */
uint64_t c3o_fmix64(uint64_t k)
{
    k ^= k >> 33;
    k *= 0xFF51AFD7ED558CCDULL;
    k ^= k >> 33;
    k *= 0xC4CEB9FE1A85EC53ULL;
    k ^= k >> 33;
    return k;
}

/* C3SIG-1 constants (this implementation's reading of H_w, Sec. 5.2). */
#define O_KEY_SEED   0x43335349472D3101ULL  /* seed of the key stream     */
#define O_TAG        0x4333534947310001ULL  /* domain tag of finalize     */
#define O_BLOCK_MUL  0x9E3779B9U            /* per-256-word block offset  */
#define O_NKEYS      258

/* Key table: K[i] = low 32 bits of the i-th SplitMix64 output. */
void c3o_keys(uint32_t *K)
{
    uint64_t st = O_KEY_SEED;
    int i;
    for (i = 0; i < O_NKEYS; i++)
        K[i] = (uint32_t)c3o_splitmix64_next(&st);
}

static uint32_t word_le(const uint8_t *b, uint64_t n, uint64_t j)
{
    /* j-th little-endian 32-bit word; bytes at or beyond n read as 0. */
    uint32_t w = 0;
    int k;
    for (k = 0; k < 4; k++) {
        uint64_t pos = 4 * j + (uint64_t)k;
        uint32_t byte = pos < n ? b[pos] : 0u;
        w |= byte << (8 * k);
    }
    return w;
}

/*
 * NH fold over the chunk's words (UMAC's NH with a Toeplitz second pass).
 * Words: D = 4 * ceil(n / 16), zero-padded.  Pair p = 2i uses keys
 * K[q..q+3], q = p mod 256, and a block offset beta = (p div 256) * 0x9E3779B9.
 */
void c3o_nh(const uint8_t *bytes, uint64_t n, const uint32_t *K,
            uint64_t *A_out, uint64_t *B_out)
{
    uint64_t D = 4 * ((n + 15) / 16);
    uint64_t A = 0, B = 0, p;
    for (p = 0; p < D; p += 2) {
        uint32_t q = (uint32_t)(p % 256);
        uint32_t beta = (uint32_t)(p / 256) * O_BLOCK_MUL;
        uint32_t m0 = word_le(bytes, n, p);
        uint32_t m1 = word_le(bytes, n, p + 1);
        uint32_t a0 = m0 + K[q] + beta;
        uint32_t a1 = m1 + K[q + 1] + beta;
        uint32_t b0 = m0 + K[q + 2] + beta;
        uint32_t b1 = m1 + K[q + 3] + beta;
        A += (uint64_t)a0 * (uint64_t)a1;
        B += (uint64_t)b0 * (uint64_t)b1;
    }
    *A_out = A;
    *B_out = B;
}

/* Finalize: fmix64 chain over (tag, dtype, ndim, shape, chunk, n, A, B). */
uint64_t c3o_finalize(int dtype, int ndim, const int64_t *shape,
                      uint64_t chunk_in_tensor, uint64_t n, uint64_t A, uint64_t B)
{
    uint64_t h = c3o_fmix64(O_TAG ^ ((uint64_t)(uint32_t)dtype << 32) ^ (uint64_t)(uint32_t)ndim);
    int d;
    for (d = 0; d < ndim; d++)
        h = c3o_fmix64(h ^ (uint64_t)shape[d]);
    h = c3o_fmix64(h ^ chunk_in_tensor);
    h = c3o_fmix64(h ^ n);
    h = c3o_fmix64(h ^ A);
    h = c3o_fmix64(h ^ B);
    return h;
}

/* ------------------------------------------------------------------ */
/* Element decoding.  Exact conversion to double; classification by    */
/* the exponent field (all ones = non-finite; NaN if mantissa != 0).    */
/* ------------------------------------------------------------------ */
static int elem_size(int dtype)
{
    switch (dtype) {
    case O_F32: return 4;
    case O_BF16: return 2;
    case O_F16: return 2;
    default: return 1;
    }
}

/* returns 0 finite, 1 NaN, 2 Inf; *v = exact value when finite */
static int decode(int dtype, const uint8_t *p, double *v)
{
    if (dtype == O_F32) {
        uint32_t u = (uint32_t)p[0] | ((uint32_t)p[1] << 8) |
                     ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
        uint32_t e = (u >> 23) & 0xFFu, m = u & 0x7FFFFFu;
        float f;
        if (e == 0xFFu) return m ? 1 : 2;
        memcpy(&f, &u, 4);
        *v = (double)f;
        return 0;
    }
    if (dtype == O_BF16) {
        /* bfloat16 is the upper half of an IEEE binary32 */
        uint32_t h = (uint32_t)p[0] | ((uint32_t)p[1] << 8);
        uint32_t e = (h >> 7) & 0xFFu, m = h & 0x7Fu;
        uint32_t u = h << 16;
        float f;
        if (e == 0xFFu) return m ? 1 : 2;
        memcpy(&f, &u, 4);
        *v = (double)f;
        return 0;
    }
    if (dtype == O_F16) {
        /* IEEE binary16: 1 sign, 5 exponent (bias 15), 10 mantissa bits */
        uint32_t h = (uint32_t)p[0] | ((uint32_t)p[1] << 8);
        uint32_t s = h >> 15, e = (h >> 10) & 0x1Fu, m = h & 0x3FFu;
        double mag;
        if (e == 0x1Fu) return m ? 1 : 2;
        if (e == 0) mag = ldexp((double)m, -24);               /* subnormal */
        else mag = ldexp((double)(m | 0x400u), (int)e - 25);  /* normal */
        *v = s ? -mag : mag;
        return 0;
    }
    return -1;
}

/* Neumaier (1974) compensated accumulation of x into (s, c). */
static void neumaier_add(double *s, double *c, double x)
{
    double t = *s + x;
    if (fabs(*s) >= fabs(x))
        *c += (*s - t) + x;
    else
        *c += (x - t) + *s;
    *s = t;
}

/*
 * Signature and numerical summary of one chunk (one replica's slice of one
 * tensor).  Outputs: sig, element count, NaN count, Inf count, absmax of the
 * finite elements, sum and sum of squares of the finite elements (compensated).
 * RAW chunks carry the hash only: n_elems = n bytes, counts and floats 0.
 */
void c3o_chunk_signature(const uint8_t *bytes, uint64_t n, int dtype, int ndim,
                         const int64_t *shape, uint64_t chunk_in_tensor,
                         const uint32_t *K,
                         uint64_t *sig, uint64_t *n_elems, uint32_t *nan_count,
                         uint32_t *inf_count, double *absmax, double *sum, double *sumsq)
{
    uint64_t A, B, i;
    c3o_nh(bytes, n, K, &A, &B);
    *sig = c3o_finalize(dtype, ndim, shape, chunk_in_tensor, n, A, B);
    *nan_count = 0;
    *inf_count = 0;
    *absmax = 0.0;
    *sum = 0.0;
    *sumsq = 0.0;
    if (dtype == O_RAW) {
        *n_elems = n;
        return;
    }
    {
        int es = elem_size(dtype);
        double s = 0.0, c = 0.0, q = 0.0, cq = 0.0, mx = 0.0;
        uint32_t nn = 0, ni = 0;
        *n_elems = n / (uint64_t)es;
        for (i = 0; i < *n_elems; i++) {
            double v = 0.0;
            int k = decode(dtype, bytes + i * (uint64_t)es, &v);
            if (k == 1) { nn++; continue; }
            if (k == 2) { ni++; continue; }
            if (fabs(v) > mx) mx = fabs(v);
            neumaier_add(&s, &c, v);
            neumaier_add(&q, &cq, v * v);   /* v*v is exact in fp64 here */
        }
        *nan_count = nn;
        *inf_count = ni;
        *absmax = mx;
        *sum = s + c;
        *sumsq = q + cq;
    }
}

/* ------------------------------------------------------------------ */
/* Chunk plan: each tensor is split independently into chunks of        */
/* chunk_bytes; the last chunk may be partial; an empty tensor has one  */
/* empty chunk (so its dtype and shape are still compared).             */
/* ------------------------------------------------------------------ */
static uint64_t tensor_bytes(int dtype, int ndim, const int64_t *shape)
{
    uint64_t n = 1;
    int d;
    for (d = 0; d < ndim; d++) n *= (uint64_t)shape[d];
    return n * (uint64_t)elem_size(dtype);
}

int64_t c3o_num_chunks(const int32_t *dtypes, const int32_t *ndims,
                       const int64_t *shapes /* [T][8] */, int T, uint64_t chunk_bytes)
{
    int64_t total = 0;
    int t;
    for (t = 0; t < T; t++) {
        uint64_t nb = tensor_bytes(dtypes[t], ndims[t], shapes + 8 * t);
        uint64_t c = (nb + chunk_bytes - 1) / chunk_bytes;
        total += (int64_t)(c ? c : 1);
    }
    return total;
}

/*
 * Signatures of all chunks of R replicas.  ptrs: host pointers [R][T]
 * (replica-major).  Outputs are structure-of-arrays [R][C].
 */
int c3o_signature(const uint8_t *const *ptrs, const int32_t *dtypes,
                  const int32_t *ndims, const int64_t *shapes, int T, int R,
                  uint64_t chunk_bytes,
                  uint64_t *sig, uint64_t *n_elems, uint32_t *nan_count,
                  uint32_t *inf_count, double *absmax, double *sum, double *sumsq,
                  uint32_t *tensor_id, uint32_t *chunk_id)
{
    uint32_t K[O_NKEYS];
    int64_t C = c3o_num_chunks(dtypes, ndims, shapes, T, chunk_bytes);
    int r, t;
    c3o_keys(K);
    for (r = 0; r < R; r++) {
        int64_t g = 0;
        for (t = 0; t < T; t++) {
            uint64_t nb = tensor_bytes(dtypes[t], ndims[t], shapes + 8 * t);
            uint64_t nc = (nb + chunk_bytes - 1) / chunk_bytes, k;
            if (nc == 0) nc = 1;
            for (k = 0; k < nc; k++, g++) {
                uint64_t off = k * chunk_bytes;
                uint64_t len = nb - off < chunk_bytes ? nb - off : chunk_bytes;
                int64_t o = (int64_t)r * C + g;
                if (nb == 0) len = 0;
                c3o_chunk_signature(ptrs[(size_t)r * (size_t)T + (size_t)t] + off, len,
                                    dtypes[t], ndims[t], shapes + 8 * t, k, K,
                                    &sig[o], &n_elems[o], &nan_count[o], &inf_count[o],
                                    &absmax[o], &sum[o], &sumsq[o]);
                tensor_id[o] = (uint32_t)t;
                chunk_id[o] = (uint32_t)k;
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Per-tensor signature (Sec. 5.2 evidence at the paper's granularity,  */
/* one value per tensor): the wrapping sum of the tensor's chunk        */
/* signatures, xor a domain tag, through fmix64.  Each chunk signature  */
/* already covers dtype, shape, chunk position, length and bytes, so    */
/* the sum keeps position sensitivity while allowing any reduction      */
/* order.                                                               */
/* sig and tensor_id are [R][C]; out is [R][T].                         */
/* ------------------------------------------------------------------ */
#define O_TAG_TENSOR 0x4333534947540001ULL

int c3o_tensor_signature(const uint64_t *sig, const uint32_t *tensor_id, int R, int64_t C, int T,
                         uint64_t *out)
{
    int r, t;
    int64_t c;
    for (r = 0; r < R; r++) {
        for (t = 0; t < T; t++) {
            uint64_t sum = 0;
            for (c = 0; c < C; c++)
                if (tensor_id[(int64_t)r * C + c] == (uint32_t)t)
                    sum += sig[(int64_t)r * C + c];
            out[(int64_t)r * T + t] = c3o_fmix64(O_TAG_TENSOR ^ sum);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Exact consensus, Sec. 5.3 / Algorithm 1 (Exact branch).              */
/* Evidence value of replica r at unit u is read at                     */
/*   base + u * unit_stride + r * replica_stride   (bytes).             */
/* ------------------------------------------------------------------ */
static uint64_t ev_bits(const uint8_t *base, int kind, int64_t off)
{
    if (kind == O_EV_U64 || kind == O_EV_F64) {
        uint64_t v;
        memcpy(&v, base + off, 8);
        return v;
    } else {
        uint32_t v;
        memcpy(&v, base + off, 4);
        return v;
    }
}

int c3o_vote_exact(const uint8_t *evidence, int kind, int64_t replica_stride,
                   int64_t unit_stride, int R, int64_t n_units,
                   uint8_t *status, uint64_t *bitmap /* [n_units][ceil(R/64)] */,
                   int32_t *majority_idx)
{
    int64_t u;
    const int W = bm_words(R);
    if (R < 2 || R > O_MAX_R) return -1;   /* a singleton compares nothing */
    for (u = 0; u < n_units; u++) {
        uint64_t e[O_MAX_R];
        uint64_t *B = bitmap + u * W;
        int cnt[O_MAX_R], r, j, best = 0, arg = -1;
        for (r = 0; r < R; r++)
            e[r] = ev_bits(evidence, kind, u * unit_stride + (int64_t)r * replica_stride);
        /* most frequent value and its count (lowest replica on ties) */
        for (r = 0; r < R; r++) {
            cnt[r] = 0;
            for (j = 0; j < R; j++) cnt[r] += (e[j] == e[r]);
            if (cnt[r] > best) { best = cnt[r]; arg = r; }
        }
        bm_clear(B, R);
        if (2 * best <= R) {          /* c* <= N/2: no strict majority */
            status[u] = O_INCONCLUSIVE;
            majority_idx[u] = -1;
            continue;
        }
        for (r = 0; r < R; r++)
            if (e[r] != e[arg]) bm_set(B, r);
        status[u] = bm_any(B, R) ? O_ATTRIBUTED : O_AGREE;
        majority_idx[u] = arg;
    }
    return 0;
}

/*
 * The plain definition of the exact result on raw bytes: replicas whose
 * chunk bytes are equal form a class; a class of more than R/2 members is
 * the majority.  Chunks are given as [R][C] host pointers with per-chunk
 * byte lengths (equal across replicas).
 */
int c3o_vote_bytes(const uint8_t *const *chunk_ptrs, const uint64_t *chunk_len,
                   int R, int64_t n_units,
                   uint8_t *status, uint64_t *bitmap /* [n_units][ceil(R/64)] */,
                   int32_t *majority_idx)
{
    int64_t u;
    const int W = bm_words(R);
    if (R < 2 || R > O_MAX_R) return -1;   /* a singleton compares nothing */
    for (u = 0; u < n_units; u++) {
        uint64_t *B = bitmap + u * W;
        int cnt[O_MAX_R], r, j, best = 0, arg = -1;
        uint64_t len = chunk_len[u];
        for (r = 0; r < R; r++) {
            const uint8_t *pr = chunk_ptrs[(int64_t)r * n_units + u];
            cnt[r] = 0;
            for (j = 0; j < R; j++) {
                const uint8_t *pj = chunk_ptrs[(int64_t)j * n_units + u];
                cnt[r] += (len == 0 || memcmp(pr, pj, len) == 0);
            }
            if (cnt[r] > best) { best = cnt[r]; arg = r; }
        }
        bm_clear(B, R);
        if (2 * best <= R) {
            status[u] = O_INCONCLUSIVE;
            majority_idx[u] = -1;
            continue;
        }
        {
            const uint8_t *pa = chunk_ptrs[(int64_t)arg * n_units + u];
            for (r = 0; r < R; r++) {
                const uint8_t *pr = chunk_ptrs[(int64_t)r * n_units + u];
                if (len != 0 && memcmp(pr, pa, len) != 0) bm_set(B, r);
            }
        }
        status[u] = bm_any(B, R) ? O_ATTRIBUTED : O_AGREE;
        majority_idx[u] = arg;
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Statistical consensus, Sec. 5.4 / Algorithm 1 (Statistical branch).  */
/* ------------------------------------------------------------------ */
static void sort_doubles(double *a, int n)
{
    int i, j;
    for (i = 1; i < n; i++) {
        double x = a[i];
        for (j = i - 1; j >= 0 && a[j] > x; j--) a[j + 1] = a[j];
        a[j + 1] = x;
    }
}

/* median of a sorted array: middle element, or the mean of the two middle */
static double median_sorted(const double *s, int n)
{
    if (n % 2 == 1) return s[(n - 1) / 2];
    return (s[n / 2 - 1] + s[n / 2]) * 0.5;
}

/* Hyndman-Fan type-7 quantile of a sorted array */
static double quantile7(const double *s, int n, double p)
{
    double h = (double)(n - 1) * p;
    int lo = (int)floor(h);
    double frac = h - (double)lo;
    if (lo + 1 >= n) return s[n - 1];
    return s[lo] + frac * (s[lo + 1] - s[lo]);
}

int c3o_vote_statistical(const uint8_t *evidence, int kind, int64_t replica_stride,
                         int64_t unit_stride, int R, int64_t n_units, double kappa,
                         uint8_t *status, uint64_t *bitmap /* [n_units][ceil(R/64)] */,
                         int32_t *majority_idx)
{
    int64_t u;
    const int W = bm_words(R);
    if (R < 2 || R > O_MAX_R) return -1;   /* a singleton compares nothing */
    for (u = 0; u < n_units; u++) {
        double tau[O_MAX_R], s[O_MAX_R], dev[O_MAX_R], devs[O_MAX_R], m, d, thr;
        int fin[O_MAX_R], r, nf = 0, k, lowmed;
        uint64_t *B = bitmap + u * W;
        bm_clear(B, R);
        for (r = 0; r < R; r++) {
            int64_t off = u * unit_stride + (int64_t)r * replica_stride;
            if (kind == O_EV_F32) {
                float f;
                memcpy(&f, evidence + off, 4);
                tau[r] = (double)f;
            } else {
                memcpy(&tau[r], evidence + off, 8);
            }
            fin[r] = isfinite(tau[r]) ? 1 : 0;
            if (fin[r]) s[nf++] = tau[r];
            else bm_set(B, r);       /* a non-finite timing is an outlier */
        }
        if (2 * nf <= R) {            /* finite values are not a majority */
            status[u] = O_INCONCLUSIVE;
            bm_clear(B, R);
            majority_idx[u] = -1;
            continue;
        }
        sort_doubles(s, nf);
        m = median_sorted(s, nf);
        k = 0;
        for (r = 0; r < R; r++)
            if (fin[r]) { dev[r] = fabs(tau[r] - m); devs[k++] = dev[r]; }
        sort_doubles(devs, nf);
        d = median_sorted(devs, nf);                                  /* MAD */
        if (d == 0.0) d = (quantile7(s, nf, 0.75) - quantile7(s, nf, 0.25)) * 0.5; /* IQR/2 */
        if (d == 0.0) d = (s[nf - 1] - s[0]) / (double)nf;           /* range/N */
        if (d != 0.0) {
            thr = kappa * d;
            for (r = 0; r < R; r++)
                if (fin[r] && dev[r] > thr) bm_set(B, r);
        }
        /* lower-median replica: the finite replica at sorted position
         * (nf-1)/2, ties broken by the lower replica index */
        lowmed = -1;
        {
            double target = s[(nf - 1) / 2];
            int before = 0;
            for (r = 0; r < R; r++)
                if (fin[r] && tau[r] < target) before++;
            /* among replicas equal to target, take the one whose stable rank
             * is (nf-1)/2 */
            for (r = 0; r < R; r++) {
                if (fin[r] && tau[r] == target) {
                    if (before == (nf - 1) / 2) { lowmed = r; break; }
                    before++;
                }
            }
        }
        status[u] = bm_any(B, R) ? O_ATTRIBUTED : O_AGREE;
        majority_idx[u] = lowmed;
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Localization: every set bitmap bit, in (unit asc, replica asc) order; */
/* the undecided (Inconclusive) units in ascending order.                */
/* ------------------------------------------------------------------ */
int c3o_localize(const uint8_t *status,
                 const uint64_t *bitmap /* [n_units][ceil(R/64)] */,
                 const int32_t *majority_idx, int R, int64_t n_units,
                 int64_t *out_unit, int32_t *out_replica, int32_t *out_majority, int64_t out_cap,
                 int64_t *undecided, int64_t und_cap, int64_t *counts)
{
    int64_t u, no = 0, nu = 0, na = 0;
    int r;
    const int W = bm_words(R);
    if (R < 2 || R > O_MAX_R) return -1;   /* a singleton compares nothing */
    for (u = 0; u < n_units; u++) {
        const uint64_t *B = bitmap + u * W;
        if (status[u] == O_INCONCLUSIVE) {
            if (nu < und_cap) undecided[nu] = u;
            nu++;
            continue;
        }
        if (!bm_any(B, R)) continue;
        na++;
        for (r = 0; r < R; r++) {
            if (bm_test(B, r)) {
                if (no < out_cap) {
                    out_unit[no] = u;
                    out_replica[no] = r;
                    out_majority[no] = majority_idx[u];
                }
                no++;
            }
        }
    }
    counts[0] = no;
    counts[1] = nu;
    counts[2] = na;
    return 0;
}

/* ------------------------------------------------------------------ */
/* Temporal confirmation over T consecutive iterations of G groups of R  */
/* ranks; rank = r * G + g.  A rank is a confirmed straggler when it is  */
/* flagged in more than half of some window of W consecutive iterations  */
/* (W capped at T); it is a protocol outlier when its fingerprint is     */
/* attributed in any iteration.  Per-rank outputs:                        */
/*   flags bit0 straggler, bit1 protocol outlier, bit2 flagged in two     */
/*   consecutive iterations at least once;                                */
/*   first_div: first attributed fingerprint iteration or -1;             */
/*   div_count, slow_count, max_window, first_window (or -1).             */
/* ------------------------------------------------------------------ */
int c3o_confirm(const uint64_t *fp_bitmap /* [T][G] */, const uint64_t *time_bitmap /* [T][G] */,
                int R, int64_t G, int64_t T, int W,
                uint32_t *flags, int32_t *first_div, uint32_t *div_count,
                uint32_t *slow_count, uint32_t *max_window, int32_t *first_window)
{
    int64_t g, t;
    int r;
    int64_t Wt = (int64_t)W < T ? (int64_t)W : T;
    if (R < 2 || R > 64 || W < 1) return -1;   /* one-word bitmaps; no singleton */
    for (r = 0; r < R; r++) {
        for (g = 0; g < G; g++) {
            int64_t rank = (int64_t)r * G + g;
            uint32_t fl = 0, dc = 0, sc = 0, mw = 0;
            int32_t fd = -1, fw = -1;
            int prev = 0;
            for (t = 0; t < T; t++) {
                int dv = (int)((fp_bitmap[t * G + g] >> r) & 1ULL);
                int sl = (int)((time_bitmap[t * G + g] >> r) & 1ULL);
                if (dv) { if (fd < 0) fd = (int32_t)t; dc++; }
                if (sl) { sc++; if (prev) fl |= 4u; }
                prev = sl;
            }
            if (Wt > 0) {
                int64_t s0;
                for (s0 = 0; s0 + Wt <= T; s0++) {
                    uint32_t c = 0;
                    for (t = s0; t < s0 + Wt; t++)
                        c += (uint32_t)((time_bitmap[t * G + g] >> r) & 1ULL);
                    if (c > mw) mw = c;
                    if (2 * (int64_t)c > Wt && fw < 0) fw = (int32_t)s0;
                }
            }
            if (fw >= 0) fl |= 1u;
            if (fd >= 0) fl |= 2u;
            flags[rank] = fl;
            first_div[rank] = fd;
            div_count[rank] = dc;
            slow_count[rank] = sc;
            max_window[rank] = mw;
            first_window[rank] = fw;
        }
    }
    return 0;
}
