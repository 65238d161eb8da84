/*
 * fp64 CPU oracle for thin-key ("asymmetric") attention.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the CPU-baseline
 * leg of the benchmark may load this library. It shares no code, header, table
 * or helper with the GPU library and never touches a device.
 *
 * What it computes is the plain definition of the method's attention core
 * (Sec. 2.1, Eq. 1-4): per head, scores over the r-wide query/key width, a
 * softmax over the visible keys, and a weighted sum of the full-width value
 * rows. The weights are scalars, so the value width d_v is independent of r
 * (the remark after Eq. 4). For every (batch b, query head h, query row i):
 *
 *     g     = h / (H_q / H_kv)                        consecutive GQA grouping
 *     last  = L - 1, or i + (S_k - S_q) when causal     bottom-right alignment
 *     s_j   = scale * sum_c Q[b,h,i,c] * K[b,g,j,c]      j = 0..last
 *     m     = max_j s_j
 *     p_j   = exp(s_j - m),   l = sum_j p_j
 *     O[b,h,i,:] = sum_j (p_j / l) * V[b,g,j,:]
 *
 * Everything is evaluated in fp64 from the exact widening of the inputs the GPU
 * receives (fp32, bf16, or OCP E4M3FN or 4-bit integer key codes times an fp32
 * per-token scale, which is the composition with quantisation the discussion in
 * Sec. 6 proposes).
 * Two passes (maximum, then sums) - no online rescaling, no blocking, no
 * splitting. Paged caches are read by explicit index through the block table.
 * A row with no visible key (decode with ctx_len 0) yields zeros.
 *
 * Parity of the functions here is pinned by the CPU tests: reduction to standard
 * attention when r = d_v (torch SDPA and a textbook formula), query absorption of
 * a factored key projection (Eq. 6-7), softmax/causality invariants, closed forms,
 * a pure-Python brute force on tiny inputs, and the E4M3 decode against torch's
 * float8_e4m3fn for all 256 codes.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { TKO_F64 = 0, TKO_F32 = 1, TKO_BF16 = 2, TKO_E4M3 = 3, TKO_INT4 = 4 };

/* OCP 8-bit floating point, E4M3FN: 1 sign bit, 4 exponent bits (bias 7),
 * 3 mantissa bits; exponent field 0 is subnormal (2^-6 * m/8); no infinities;
 * S.1111.111 is NaN; largest finite magnitude 1.75 * 2^8 = 448. */
double tko_e4m3_value(uint8_t code) {
    int s = code >> 7, e = (code >> 3) & 15, m = code & 7;
    double mag;
    if (e == 15 && m == 7) return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, -6);
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return s ? -mag : mag;
}

/* 4-bit integer key codes, excess-8: the nibble n holds the integer n - 8
 * (-7 .. 7 in use); entry i of a row is nibble i % 2 (low nibble first) of byte
 * i / 2. Rows have an even number of entries, so they start on byte boundaries. */
double tko_int4_value(const uint8_t* codes, size_t i) {
    const uint8_t byte = codes[i >> 1];
    const int n = (i & 1) ? (byte >> 4) : (byte & 15);
    return (double)(n - 8);
}

/* bfloat16 is the upper half of an IEEE binary32. */
static double bf16_value(uint16_t bits) {
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

/* Element i of a typed array, widened exactly to fp64. */
static double ld(const void* p, int dt, size_t i) {
    switch (dt) {
        case TKO_F64: return ((const double*)p)[i];
        case TKO_F32: return (double)((const float*)p)[i];
        case TKO_BF16: return bf16_value(((const uint16_t*)p)[i]);
        case TKO_E4M3: return tko_e4m3_value(((const uint8_t*)p)[i]);
        case TKO_INT4: return tko_int4_value((const uint8_t*)p, i);
        default: return NAN;
    }
}

/* One query row against keys/values given by a row-address callback. */
typedef struct {
    const void* K; int k_dt; const float* k_scale;
    const void* V; int v_dt;
    long r, dv;
    /* row index of key/value j in the K (and V, scale) arrays */
    const int64_t* rows;
} kv_view;

static void attend_row(const double* q, const kv_view* kv, long n_keys, double scale,
                       double* s, double* out) {
    long dv = kv->dv, r = kv->r;
    for (long c = 0; c < dv; c++) out[c] = 0.0;
    if (n_keys <= 0) return;
    /* scores */
    for (long j = 0; j < n_keys; j++) {
        int64_t row = kv->rows[j];
        double ks = kv->k_scale ? (double)kv->k_scale[row] : 1.0;
        double acc = 0.0;
        for (long c = 0; c < r; c++) acc += q[c] * (ld(kv->K, kv->k_dt, (size_t)row * r + c) * ks);
        s[j] = scale * acc;
    }
    /* softmax: maximum, exponentials, normaliser */
    double m = -INFINITY;
    for (long j = 0; j < n_keys; j++) m = s[j] > m ? s[j] : m;
    double l = 0.0;
    for (long j = 0; j < n_keys; j++) {
        s[j] = exp(s[j] - m);
        l += s[j];
    }
    /* weighted sum of the full-width value rows */
    for (long j = 0; j < n_keys; j++) {
        int64_t row = kv->rows[j];
        double w = s[j] / l;
        for (long c = 0; c < dv; c++) out[c] += w * ld(kv->V, kv->v_dt, (size_t)row * dv + c);
    }
}

static int set_threads(int threads) {
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
    return omp_get_max_threads();
#else
    (void)threads;
    return 1;
#endif
}

int tko_max_threads(void) { return set_threads(0); }

/*
 * Prefill / full attention.
 * Q [B,Hq,Sq,r]  K [B,Hkv,Sk,r]  V [B,Hkv,Sk,dv]  O [B,Hq,Sq,dv] (fp64, written).
 * k_scale: NULL, or fp32 [B,Hkv,Sk] multiplying each key row (E4M3 keys).
 * causal: query row i sees keys 0..i+(Sk-Sq). Returns 0, or -1 on bad shapes.
 */
int tko_prefill(const void* Q, int q_dt, const void* K, int k_dt, const float* k_scale,
                const void* V, int v_dt, double* O,
                long B, long Hq, long Hkv, long Sq, long Sk, long r, long dv,
                int causal, double scale, int threads) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || Sq < 0 || Sk < 0 || r <= 0 || dv <= 0) return -1;
    if (causal && Sq > Sk) return -1;
    long G = Hq / Hkv;
    set_threads(threads);
    long n_rows = B * Hq * Sq;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)(Sk > 0 ? Sk : 1));
        double* q = (double*)malloc(sizeof(double) * (size_t)r);
        int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)(Sk > 0 ? Sk : 1));
#pragma omp for schedule(dynamic, 16)
        for (long idx = 0; idx < n_rows; idx++) {
            long i = idx % Sq, h = (idx / Sq) % Hq, b = idx / (Sq * Hq);
            long g = h / G;
            long n_keys = causal ? i + (Sk - Sq) + 1 : Sk;
            for (long c = 0; c < r; c++) q[c] = ld(Q, q_dt, (size_t)idx * r + c);
            for (long j = 0; j < n_keys; j++) rows[j] = (b * Hkv + g) * Sk + j;
            kv_view kv = {K, k_dt, k_scale, V, v_dt, r, dv, rows};
            attend_row(q, &kv, n_keys, scale, s, O + (size_t)idx * dv);
        }
        free(s);
        free(q);
        free(rows);
    }
    return 0;
}

/*
 * Single-token decode against a thin-key / full-value cache.
 * Q [B,Hq,r]; O [B,Hq,dv] (fp64, written).
 * contiguous (block_table == NULL): K [B,Hkv,max_ctx,r], V [B,Hkv,max_ctx,dv],
 *     k_scale [B,Hkv,max_ctx].
 * paged: K [nblk,Hkv,bs,r], V [nblk,Hkv,bs,dv], k_scale [nblk,Hkv,bs];
 *     token t of sequence b sits in block block_table[b*max_blocks + t/bs], slot t%bs.
 * Query (b,h) attends to all ctx_lens[b] cached tokens (the newest is already in).
 */
int tko_decode(const void* Q, int q_dt, const void* K, int k_dt, const float* k_scale,
               const void* V, int v_dt, double* O,
               long B, long Hq, long Hkv, const int32_t* ctx_lens, long max_ctx, long r, long dv,
               double scale, const int32_t* block_table, long block_size, long max_blocks,
               int threads) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || r <= 0 || dv <= 0 || max_ctx < 0) return -1;
    if (block_table && (block_size <= 0 || max_blocks <= 0)) return -1;
    for (long b = 0; b < B; b++) {
        if (ctx_lens[b] < 0) return -1;
        if (!block_table && ctx_lens[b] > max_ctx) return -1;
        if (block_table && ctx_lens[b] > block_size * max_blocks) return -1;
    }
    long G = Hq / Hkv;
    set_threads(threads);
    long n_rows = B * Hq;
    long cap = 1;
    for (long b = 0; b < B; b++) cap = ctx_lens[b] > cap ? ctx_lens[b] : cap;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)cap);
        double* q = (double*)malloc(sizeof(double) * (size_t)r);
        int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
#pragma omp for schedule(dynamic, 1)
        for (long idx = 0; idx < n_rows; idx++) {
            long h = idx % Hq, b = idx / Hq, g = h / G;
            long L = ctx_lens[b];
            for (long c = 0; c < r; c++) q[c] = ld(Q, q_dt, (size_t)idx * r + c);
            for (long t = 0; t < L; t++) {
                if (block_table) {
                    int64_t blk = block_table[b * max_blocks + t / block_size];
                    rows[t] = (blk * Hkv + g) * block_size + t % block_size;
                } else {
                    rows[t] = (b * Hkv + g) * max_ctx + t;
                }
            }
            kv_view kv = {K, k_dt, k_scale, V, v_dt, r, dv, rows};
            attend_row(q, &kv, L, scale, s, O + (size_t)idx * dv);
        }
        free(s);
        free(q);
        free(rows);
    }
    return 0;
}

/*
 * Gradients of the causal (or full) prefill attention with respect to Q, K and
 * V, for the thin-key training path (the paper trains thin-key models from
 * scratch, Sec. 3). Written from the chain rule through the definition above,
 * with the GQA grouping g = h / (H_q / H_kv):
 *
 *     P[h,i,j]  = exp(s[h,i,j] - lse[h,i]),  lse[h,i] = log sum_j exp(s[h,i,j])
 *     dP[h,i,j] = sum_c dO[h,i,c] * V[g,j,c]
 *     D[h,i]    = sum_j P[h,i,j] * dP[h,i,j]
 *     dS[h,i,j] = P[h,i,j] * (dP[h,i,j] - D[h,i])
 *     dQ[h,i,:] = scale * sum_j dS[h,i,j] * K[g,j,:]
 *     dK[g,j,:] = scale * sum_{h in g} sum_i dS[h,i,j] * Q[h,i,:]
 *     dV[g,j,:] = sum_{h in g} sum_i P[h,i,j] * dO[h,i,:]
 *
 * D is the sum of P * dP over the row, which equals the sum of dO * O for the
 * exact forward output O. When O is given (not NULL), D is instead taken as
 * sum_c dO[h,i,c] * O[h,i,c] of that O: the form of the backward pass that is
 * handed the forward output as stored (rounded), which then enters D, and
 * through D the query and key gradients. Phase 1 goes row by row (lse, D, dQ),
 * phase 2 key row by key row (dK, dV), recomputing scores as needed, all in
 * fp64 from the exact widening of the inputs.
 *
 * Only query rows i >= row_lo are processed: dQ and lse of those rows are
 * exact, and dK, dV hold the contributions of those rows only, which for a
 * causal mask is the whole gradient of keys j >= row_lo + (Sk - Sq). row_lo = 0
 * gives the full gradients. dQ [B,Hq,Sq,r], dK [B,Hkv,Sk,r], dV [B,Hkv,Sk,dv],
 * lse [B,Hq,Sq] (natural logarithm) are fp64 and written (rows below row_lo of
 * dQ and lse are left untouched). Returns 0, or -1 on bad shapes.
 */
int tko_prefill_backward(const void* Q, int q_dt, const void* K, int k_dt, const void* V, int v_dt,
                         const void* dO, int do_dt, const void* O, int o_dt, double* dQ, double* dK, double* dV,
                         double* lse,
                         long B, long Hq, long Hkv, long Sq, long Sk, long r, long dv,
                         int causal, double scale, long row_lo, int threads) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || Sq < 0 || Sk <= 0 || r <= 0 || dv <= 0) return -1;
    if ((causal && Sq > Sk) || row_lo < 0) return -1;
    const long G = Hq / Hkv, off = Sk - Sq;
    set_threads(threads);
    double* Dr = (double*)malloc(sizeof(double) * (size_t)(B * Hq * (Sq > 0 ? Sq : 1)));
    if (!Dr) return -1;

    /* phase 1: per query row, the log-sum-exp, D and dQ */
    const long n_rows = B * Hq * Sq;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)Sk);
        double* dp = (double*)malloc(sizeof(double) * (size_t)Sk);
#pragma omp for schedule(dynamic, 8)
        for (long idx = 0; idx < n_rows; idx++) {
            const long i = idx % Sq, h = (idx / Sq) % Hq, b = idx / (Sq * Hq), g = h / G;
            if (i < row_lo) continue;
            const long n = causal ? i + off + 1 : Sk;
            const size_t kv0 = (size_t)(b * Hkv + g) * Sk;
            double m = -INFINITY;
            for (long j = 0; j < n; j++) {
                double acc = 0.0;
                for (long c = 0; c < r; c++)
                    acc += ld(Q, q_dt, (size_t)idx * r + c) * ld(K, k_dt, (kv0 + j) * r + c);
                s[j] = acc * scale;
                if (s[j] > m) m = s[j];
            }
            double l = 0.0;
            for (long j = 0; j < n; j++) l += exp(s[j] - m);
            const double ls = m + log(l);
            lse[idx] = ls;
            double D = 0.0;
            for (long j = 0; j < n; j++) {
                double acc = 0.0;
                for (long c = 0; c < dv; c++)
                    acc += ld(dO, do_dt, (size_t)idx * dv + c) * ld(V, v_dt, (kv0 + j) * dv + c);
                dp[j] = acc;
                s[j] = exp(s[j] - ls); /* now P */
                D += s[j] * dp[j];
            }
            if (O) {
                D = 0.0;
                for (long c = 0; c < dv; c++)
                    D += ld(dO, do_dt, (size_t)idx * dv + c) * ld(O, o_dt, (size_t)idx * dv + c);
            }
            Dr[idx] = D;
            for (long c = 0; c < r; c++) dQ[(size_t)idx * r + c] = 0.0;
            for (long j = 0; j < n; j++) {
                const double ds = s[j] * (dp[j] - D);
                for (long c = 0; c < r; c++) dQ[(size_t)idx * r + c] += scale * ds * ld(K, k_dt, (kv0 + j) * r + c);
            }
        }
        free(s);
        free(dp);
    }

    /* phase 2: per key row, dK and dV summed over the group's heads and rows */
    const long n_keys = B * Hkv * Sk;
#pragma omp parallel for schedule(dynamic, 8)
    for (long kidx = 0; kidx < n_keys; kidx++) {
        const long j = kidx % Sk, g = (kidx / Sk) % Hkv, b = kidx / (Sk * Hkv);
        double* dk = dK + (size_t)kidx * r;
        double* dvv = dV + (size_t)kidx * dv;
        for (long c = 0; c < r; c++) dk[c] = 0.0;
        for (long c = 0; c < dv; c++) dvv[c] = 0.0;
        long i0 = causal ? j - off : 0;
        if (i0 < row_lo) i0 = row_lo;
        if (i0 < 0) i0 = 0;
        for (long h = g * G; h < (g + 1) * G; h++) {
            for (long i = i0; i < Sq; i++) {
                const size_t idx = (size_t)((b * Hq + h) * Sq + i);
                double acc = 0.0;
                for (long c = 0; c < r; c++) acc += ld(Q, q_dt, idx * r + c) * ld(K, k_dt, (size_t)kidx * r + c);
                const double p = exp(scale * acc - lse[idx]);
                double dpv = 0.0;
                for (long c = 0; c < dv; c++) dpv += ld(dO, do_dt, idx * dv + c) * ld(V, v_dt, (size_t)kidx * dv + c);
                const double ds = p * (dpv - Dr[idx]);
                for (long c = 0; c < r; c++) dk[c] += scale * ds * ld(Q, q_dt, idx * r + c);
                for (long c = 0; c < dv; c++) dvv[c] += p * ld(dO, do_dt, idx * dv + c);
            }
        }
    }
    free(Dr);
    return 0;
}
