/*
 * WhiteMatter CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 statement of what the WhiteMatter cross-layer KV pool
 * and the per-layer channel attention compute, written from the paper
 * ("WhiteMatter: All-to-All Cross-Layer Connections via KV Mixing"):
 *   Section 3.1 Step 1 (pre-mix RMSNorm, layer-subsampled linear router, mix),
 *   Section 3.1 Step 2 (mid RMSNorm, per-channel K/V projection, key norm, RoPE),
 *   Section 3.1 Step 3 (fixed per-layer channel selection, causal SDPA),
 *   Section 3.1 "Router initialization" (bias patterns),
 *   Section 3.2 (decode: the learned dummy KV slot that keeps a token's queries
 *                off its own channels).
 * The query side is the unchanged Qwen3 block of Section 4.1 (input RMSNorm,
 * W^Q, per-head q-norm, RoPE).
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library. It shares no code, header or table with the GPU library.
 * Every value is carried in double; inputs are the exact values the GPU sees.
 * Loops follow the definitions directly: no blocking, no fusion, no reordering
 * beyond what a definition states. OpenMP only splits independent tokens/rows.
 *
 * Conventions the paper leaves open (each one is a documented reading):
 *   - RMSNorm(x) = g * x / sqrt(mean(x^2) + eps)                (Qwen3 style)
 *   - router input: the normed states of layers {L-1-p*m}, stacked in
 *     ascending layer order; reshape of the kL router output is row-major,
 *     alpha[j][l] = a[j*L + l]
 *   - key norm gain g_knorm[j] has length d and is shared by the KV heads
 *   - RoPE is the rotate-half form: pair (m, m + d/2) is rotated by
 *     pos * theta^(-2m/d); pos(i) = position of the token in its sequence
 *   - the dummy K/V of channel c and KV head h is used verbatim (no norm, no
 *     RoPE); paper mask: a query at position t sees the dummy and slots s < t;
 *     inclusive mask: slots s <= t and no dummy
 *   - softmax-over-depth mix mode (optional): alpha[j][.] <- softmax over l
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define WMO_MIX_LINEAR 0
#define WMO_MIX_SOFTMAX 1
#define WMO_MASK_PAPER 0
#define WMO_MASK_INCLUSIVE 1
/* Router variants (Section 5.3, ablation studies): the paper's content-dependent router;
 * static learnable mixing weights (alpha = b, no router); no deep-to-shallow feedback
 * (k = L, channel j is built from source layers 0..j only, its router reading only
 * those layers). */
#define WMO_ROUTER_DYNAMIC 0
#define WMO_ROUTER_STATIC 1
#define WMO_ROUTER_NOFEEDBACK 2

typedef struct {
    int B, T_new, L, k, D, Hq, Hkv, d, p, S_cap;
    int mix_mode, mask_mode, router_mode;
    double eps, rope_theta;
} wmo_dims;

/* All parameters as double arrays, row-major, shapes as named. */
typedef struct {
    const double *g_pre;   /* [2][L][D]       pre-mix RMSNorm gains, K then V   */
    const double *W_alpha; /* [2][k*L][L'*D]  router weights, K then V          */
    const double *b_alpha; /* [2][k*L]        router biases                      */
    const double *g_mid;   /* [2][k][D]       mid RMSNorm gains per channel     */
    const double *Wk;      /* [k][Hkv*d][D]   key projection per channel        */
    const double *Wv;      /* [k][Hkv*d][D]   value projection per channel      */
    const double *g_knorm; /* [k][d]          key-norm gain per channel         */
    const double *Kd;      /* [k][Hkv][d]     dummy key per channel, KV head    */
    const double *Vd;      /* [k][Hkv][d]     dummy value                       */
    const double *g_in;    /* [L][D]          consumer input RMSNorm gains      */
    const double *Wq;      /* [L][Hq*d][D]    consumer query projections        */
    const double *g_qnorm; /* [L][d]          consumer q-norm gains             */
} wmo_params;

/* ---------------------------------------------------------------- basics */

/* RMSNorm, Section 3.1 Step 1 ("each source state is first RMS-normalized")
 * and Step 2; y = g * x / sqrt(mean(x^2) + eps). */
void wmo_rmsnorm(const double *x, const double *g, int n, double eps, double *y)
{
    double ss = 0.0;
    for (int e = 0; e < n; ++e)
        ss += x[e] * x[e];
    double inv = 1.0 / sqrt(ss / (double)n + eps);
    for (int e = 0; e < n; ++e)
        y[e] = g[e] * x[e] * inv;
}

/* Rotary position embedding, rotate-half form, in place on x[0..d). */
void wmo_rope(double *x, int d, double pos, double theta)
{
    int half = d / 2;
    for (int m = 0; m < half; ++m) {
        double freq = pow(theta, -2.0 * (double)m / (double)d);
        double ang = pos * freq;
        double c = cos(ang), s = sin(ang);
        double a = x[m], b = x[m + half];
        x[m] = a * c - b * s;
        x[m + half] = b * c + a * s;
    }
}

/* Number of router inputs L' = ceil(L/p), Section 3.1 Step 1. */
int wmo_router_inputs(int L, int p)
{
    return (L + p - 1) / p;
}

/* The layers the router reads: every p-th layer counting down from L-1,
 * returned in ascending order (the stacking order of xi). */
void wmo_router_layers(int L, int p, int *sel)
{
    int Lp = wmo_router_inputs(L, p);
    for (int m = 0; m < Lp; ++m)
        sel[Lp - 1 - m] = L - 1 - p * m;
}

/* Router bias initialisation, Section 3.1 "Router initialization":
 * k = 1 -> top layer; 1 < k < L -> layer l feeds channel l mod k;
 * k = L -> channel j takes layer min(j+1, L-1). b has k*L entries, read as
 * alpha[j][l] = b[j*L + l]. Returns 0, or -1 for k outside [1, L]. */
int wmo_init_bias(int L, int k, double *b)
{
    if (k < 1 || k > L)
        return -1;
    for (int i = 0; i < k * L; ++i)
        b[i] = 0.0;
    if (k == 1) {
        b[L - 1] = 1.0;
    } else if (k < L) {
        for (int l = 0; l < L; ++l)
            b[(l % k) * L + l] = 1.0;
    } else {
        for (int j = 0; j < k; ++j) {
            int src = j + 1 < L - 1 ? j + 1 : L - 1;
            b[j * L + src] = 1.0;
        }
    }
    return 0;
}

/* Inverse of the consumer -> channel map, Section 3.1 Step 3: channel c is
 * read by members[offsets[c] .. offsets[c+1]) in ascending layer order.
 * Returns 0, or -1 if a map entry is outside [0, k). */
int wmo_channel_groups(int L, int k, const int *map, int *offsets, int *members)
{
    for (int l = 0; l < L; ++l)
        if (map[l] < 0 || map[l] >= k)
            return -1;
    int pos = 0;
    for (int c = 0; c < k; ++c) {
        offsets[c] = pos;
        for (int l = 0; l < L; ++l)
            if (map[l] == c)
                members[pos++] = l;
    }
    offsets[k] = pos;
    return 0;
}

/* ----------------------------------------------------- Step 1: the mix */

/* One token: L states h[L][D] -> mixing weights alpha[2][k][L] and mixed
 * channels mixed[2][k][D] (Section 3.1 Step 1, both branches). */
void wmo_pool_mix_token(const wmo_dims *dm, const wmo_params *P, const double *h,
                        double *alpha, double *mixed)
{
    int L = dm->L, k = dm->k, D = dm->D;
    int Lp = wmo_router_inputs(L, dm->p);
    int *sel = (int *)malloc(sizeof(int) * Lp);
    double *hn = (double *)malloc(sizeof(double) * L * D);
    wmo_router_layers(L, dm->p, sel);

    for (int br = 0; br < 2; ++br) {
        /* pre-mix RMSNorm of every source state */
        for (int l = 0; l < L; ++l)
            wmo_rmsnorm(h + (size_t)l * D, P->g_pre + ((size_t)br * L + l) * D, D,
                        dm->eps, hn + (size_t)l * D);
        /* linear router on the stacked selected states, then reshape k x L */
        const double *W = P->W_alpha + (size_t)br * k * L * Lp * D;
        const double *bias = P->b_alpha + (size_t)br * k * L;
        double *al = alpha + (size_t)br * k * L;
        int nofb = dm->router_mode == WMO_ROUTER_NOFEEDBACK;
        for (int o = 0; o < k * L; ++o) {
            int j = o / L;
            double a = bias[o];
            if (dm->router_mode != WMO_ROUTER_STATIC) {
                for (int m = 0; m < Lp; ++m) {
                    if (nofb && sel[m] > j)
                        continue; /* channel j's router reads source layers <= j only */
                    const double *x = hn + (size_t)sel[m] * D;
                    const double *w = W + (size_t)o * Lp * D + (size_t)m * D;
                    for (int e = 0; e < D; ++e)
                        a += w[e] * x[e];
                }
            }
            al[o] = a; /* alpha[j][l] with o = j*L + l */
        }
        /* sources a channel may mix: all L, or 0..j without feedback */
        for (int j = 0; j < k; ++j) {
            int nl = nofb ? j + 1 : L;
            double *row = al + (size_t)j * L;
            if (dm->mix_mode == WMO_MIX_SOFTMAX) {
                double mx = row[0], s = 0.0;
                for (int l = 1; l < nl; ++l)
                    if (row[l] > mx)
                        mx = row[l];
                for (int l = 0; l < nl; ++l)
                    s += exp(row[l] - mx);
                for (int l = 0; l < nl; ++l)
                    row[l] = exp(row[l] - mx) / s;
            }
            for (int l = nl; l < L; ++l)
                row[l] = 0.0;
        }
        /* each channel is the alpha-weighted sum of the normed states */
        for (int j = 0; j < k; ++j) {
            double *out = mixed + ((size_t)br * k + j) * D;
            for (int e = 0; e < D; ++e) {
                double acc = 0.0;
                for (int l = 0; l < L; ++l)
                    acc += al[(size_t)j * L + l] * hn[(size_t)l * D + e];
                out[e] = acc;
            }
        }
    }
    free(hn);
    free(sel);
}

/* ---------------------------------------------- Step 2: K/V projection */

/* One token: mixed[2][k][D] -> cache rows kt[k][Hkv][d] (mid norm, W^K_j,
 * key norm, RoPE at pos) and vt[k][Hkv][d] (mid norm, W^V_j, stored raw). */
void wmo_project_token(const wmo_dims *dm, const wmo_params *P, const double *mixed,
                       double pos, double *kt, double *vt)
{
    int k = dm->k, D = dm->D, Hkv = dm->Hkv, d = dm->d, O = Hkv * d;
    double *u = (double *)malloc(sizeof(double) * D);
    double *y = (double *)malloc(sizeof(double) * O);
    for (int br = 0; br < 2; ++br) {
        const double *W = br == 0 ? P->Wk : P->Wv;
        double *dst = br == 0 ? kt : vt;
        for (int j = 0; j < k; ++j) {
            wmo_rmsnorm(mixed + ((size_t)br * k + j) * D, P->g_mid + ((size_t)br * k + j) * D,
                        D, dm->eps, u);
            const double *Wj = W + (size_t)j * O * D;
            for (int o = 0; o < O; ++o) {
                double a = 0.0;
                for (int e = 0; e < D; ++e)
                    a += Wj[(size_t)o * D + e] * u[e];
                y[o] = a;
            }
            for (int hh = 0; hh < Hkv; ++hh) {
                double *row = dst + ((size_t)j * Hkv + hh) * d;
                if (br == 0) {
                    wmo_rmsnorm(y + (size_t)hh * d, P->g_knorm + (size_t)j * d, d, dm->eps, row);
                    wmo_rope(row, d, pos, dm->rope_theta);
                } else {
                    memcpy(row, y + (size_t)hh * d, sizeof(double) * d);
                }
            }
        }
    }
    free(y);
    free(u);
}

/* ----------------------------------------------------- query side */

/* Consumer layer l, one token: q[Hq][d] = RoPE(qnorm(W^Q_l RMSNorm_in(h_l))). */
void wmo_query_token(const wmo_dims *dm, const wmo_params *P, const double *h_l, int l,
                     double pos, double *q)
{
    int D = dm->D, Hq = dm->Hq, d = dm->d, O = Hq * d;
    double *x = (double *)malloc(sizeof(double) * D);
    double *y = (double *)malloc(sizeof(double) * O);
    wmo_rmsnorm(h_l, P->g_in + (size_t)l * D, D, dm->eps, x);
    const double *W = P->Wq + (size_t)l * O * D;
    for (int o = 0; o < O; ++o) {
        double a = 0.0;
        for (int e = 0; e < D; ++e)
            a += W[(size_t)o * D + e] * x[e];
        y[o] = a;
    }
    for (int hh = 0; hh < Hq; ++hh) {
        wmo_rmsnorm(y + (size_t)hh * d, P->g_qnorm + (size_t)l * d, d, dm->eps, q + (size_t)hh * d);
        wmo_rope(q + (size_t)hh * d, d, pos, dm->rope_theta);
    }
    free(y);
    free(x);
}

/* ----------------------------------------------------- attention */

/* One query vector q[d] against nvis cached keys/values (rows strided by
 * kstride/vstride doubles), optionally preceded by a dummy slot (kd, vd;
 * kd == NULL means no dummy). Scale 1/sqrt(d), plain softmax in fp64. */
void wmo_attend_row(int d, const double *q, const double *K, long kstride, const double *V,
                    long vstride, long nvis, const double *kd, const double *vd, double *o)
{
    long n = nvis + (kd ? 1 : 0);
    double *s = (double *)malloc(sizeof(double) * (n > 0 ? n : 1));
    double scale = 1.0 / sqrt((double)d);
    long idx = 0;
    if (kd) {
        double a = 0.0;
        for (int e = 0; e < d; ++e)
            a += q[e] * kd[e];
        s[idx++] = a * scale;
    }
    for (long t = 0; t < nvis; ++t) {
        double a = 0.0;
        for (int e = 0; e < d; ++e)
            a += q[e] * K[t * kstride + e];
        s[idx++] = a * scale;
    }
    for (int e = 0; e < d; ++e)
        o[e] = 0.0;
    if (n == 0) {
        free(s);
        return;
    }
    double mx = s[0];
    for (long t = 1; t < n; ++t)
        if (s[t] > mx)
            mx = s[t];
    double z = 0.0;
    for (long t = 0; t < n; ++t) {
        s[t] = exp(s[t] - mx);
        z += s[t];
    }
    idx = 0;
    if (kd) {
        for (int e = 0; e < d; ++e)
            o[e] += s[0] * vd[e];
        idx = 1;
    }
    for (long t = 0; t < nvis; ++t, ++idx)
        for (int e = 0; e < d; ++e)
            o[e] += s[idx] * V[t * vstride + e];
    for (int e = 0; e < d; ++e)
        o[e] /= z;
    free(s);
}

/* ------------------------------------------------- whole-tensor drivers */
/* Layouts: H[B][T_new][L][D]; alpha[2][N][k][L]; mixed[2][k][N][D];
 * cache Kc, Vc[k][B][Hkv][S_cap][d]; Q[L][B][Hq][T_new][d];
 * O[L][B][T_new][Hq*d]; ctx_len[B]. Token n = b*T_new + i sits at position
 * ctx_len[b] + i and is stored at that cache slot. A NULL token/row list
 * means "all". */

static int list_len(const int *list, int nlist, int all)
{
    return list ? nlist : all;
}

void wmo_router_mix(const wmo_dims *dm, const wmo_params *P, const double *H, const int *toks,
                    int ntok, double *alpha_out, double *mixed_out)
{
    int N = dm->B * dm->T_new, L = dm->L, k = dm->k, D = dm->D;
    int cnt = list_len(toks, ntok, N);
#pragma omp parallel for schedule(dynamic)
    for (int t = 0; t < cnt; ++t) {
        int n = toks ? toks[t] : t;
        double *al = (double *)malloc(sizeof(double) * 2 * k * L);
        double *mx = (double *)malloc(sizeof(double) * 2 * k * D);
        wmo_pool_mix_token(dm, P, H + (size_t)n * L * D, al, mx);
        for (int br = 0; br < 2; ++br) {
            if (alpha_out)
                memcpy(alpha_out + ((size_t)br * N + n) * k * L, al + (size_t)br * k * L,
                       sizeof(double) * k * L);
            if (mixed_out)
                for (int j = 0; j < k; ++j)
                    memcpy(mixed_out + (((size_t)br * k + j) * N + n) * D,
                           mx + ((size_t)br * k + j) * D, sizeof(double) * D);
        }
        free(mx);
        free(al);
    }
}

static void store_cache_rows(const wmo_dims *dm, int b, long slot, const double *kt,
                             const double *vt, double *Kc, double *Vc)
{
    int k = dm->k, Hkv = dm->Hkv, d = dm->d;
    for (int j = 0; j < k; ++j)
        for (int hh = 0; hh < Hkv; ++hh) {
            size_t off = ((((size_t)j * dm->B + b) * Hkv + hh) * dm->S_cap + slot) * d;
            memcpy(Kc + off, kt + ((size_t)j * Hkv + hh) * d, sizeof(double) * d);
            memcpy(Vc + off, vt + ((size_t)j * Hkv + hh) * d, sizeof(double) * d);
        }
}

void wmo_kv_project(const wmo_dims *dm, const wmo_params *P, const double *mixed,
                    const int *ctx_len, const int *toks, int ntok, double *Kc, double *Vc)
{
    int N = dm->B * dm->T_new, k = dm->k, D = dm->D, KV = dm->k * dm->Hkv * dm->d;
    int cnt = list_len(toks, ntok, N);
#pragma omp parallel for schedule(dynamic)
    for (int t = 0; t < cnt; ++t) {
        int n = toks ? toks[t] : t;
        int b = n / dm->T_new, i = n % dm->T_new;
        long pos = (long)(ctx_len ? ctx_len[b] : 0) + i;
        double *mx = (double *)malloc(sizeof(double) * 2 * k * D);
        double *kt = (double *)malloc(sizeof(double) * KV);
        double *vt = (double *)malloc(sizeof(double) * KV);
        for (int br = 0; br < 2; ++br)
            for (int j = 0; j < k; ++j)
                memcpy(mx + ((size_t)br * k + j) * D, mixed + (((size_t)br * k + j) * N + n) * D,
                       sizeof(double) * D);
        wmo_project_token(dm, P, mx, (double)pos, kt, vt);
        store_cache_rows(dm, b, pos, kt, vt, Kc, Vc);
        free(vt);
        free(kt);
        free(mx);
    }
}

/* Steps 1 and 2 together for the listed tokens: H -> cache slots. */
void wmo_pool(const wmo_dims *dm, const wmo_params *P, const double *H, const int *ctx_len,
              const int *toks, int ntok, double *Kc, double *Vc)
{
    int N = dm->B * dm->T_new, L = dm->L, k = dm->k, D = dm->D, KV = dm->k * dm->Hkv * dm->d;
    int cnt = list_len(toks, ntok, N);
#pragma omp parallel for schedule(dynamic)
    for (int t = 0; t < cnt; ++t) {
        int n = toks ? toks[t] : t;
        int b = n / dm->T_new, i = n % dm->T_new;
        long pos = (long)(ctx_len ? ctx_len[b] : 0) + i;
        double *al = (double *)malloc(sizeof(double) * 2 * k * L);
        double *mx = (double *)malloc(sizeof(double) * 2 * k * D);
        double *kt = (double *)malloc(sizeof(double) * KV);
        double *vt = (double *)malloc(sizeof(double) * KV);
        wmo_pool_mix_token(dm, P, H + (size_t)n * L * D, al, mx);
        wmo_project_token(dm, P, mx, (double)pos, kt, vt);
        store_cache_rows(dm, b, pos, kt, vt, Kc, Vc);
        free(vt);
        free(kt);
        free(mx);
        free(al);
    }
}

/* Steps 1 and 2 for the listed tokens, returning each token's cache rows
 * Krows/Vrows[n][k][Hkv][d] (as stored at its slot) instead of a cache. */
void wmo_pool_rows(const wmo_dims *dm, const wmo_params *P, const double *H, const int *ctx_len,
                   const int *toks, int ntok, double *Krows, double *Vrows)
{
    int N = dm->B * dm->T_new, L = dm->L, k = dm->k, D = dm->D, KV = dm->k * dm->Hkv * dm->d;
    int cnt = list_len(toks, ntok, N);
#pragma omp parallel for schedule(dynamic)
    for (int t = 0; t < cnt; ++t) {
        int n = toks ? toks[t] : t;
        int b = n / dm->T_new, i = n % dm->T_new;
        long pos = (long)(ctx_len ? ctx_len[b] : 0) + i;
        double *al = (double *)malloc(sizeof(double) * 2 * k * L);
        double *mx = (double *)malloc(sizeof(double) * 2 * k * D);
        wmo_pool_mix_token(dm, P, H + (size_t)n * L * D, al, mx);
        wmo_project_token(dm, P, mx, (double)pos, Krows + (size_t)n * KV, Vrows + (size_t)n * KV);
        free(mx);
        free(al);
    }
}

void wmo_q_project(const wmo_dims *dm, const wmo_params *P, const double *H, const int *ctx_len,
                   const int *toks, int ntok, double *Q)
{
    int N = dm->B * dm->T_new, L = dm->L, D = dm->D, Hq = dm->Hq, d = dm->d, T = dm->T_new;
    int cnt = list_len(toks, ntok, N);
#pragma omp parallel for schedule(dynamic)
    for (int t = 0; t < cnt; ++t) {
        int n = toks ? toks[t] : t;
        int b = n / T, i = n % T;
        long pos = (long)(ctx_len ? ctx_len[b] : 0) + i;
        double *q = (double *)malloc(sizeof(double) * Hq * d);
        for (int l = 0; l < L; ++l) {
            wmo_query_token(dm, P, H + ((size_t)n * L + l) * D, l, (double)pos, q);
            for (int hh = 0; hh < Hq; ++hh)
                memcpy(Q + ((((size_t)l * dm->B + b) * Hq + hh) * T + i) * d, q + (size_t)hh * d,
                       sizeof(double) * d);
        }
        free(q);
    }
}

/* Step 3: consumer l reads channel map[l]. A row r = (l*B + b)*T_new + i
 * produces O[l][b][i][0 .. Hq*d).
 * Document mask (Section 4.1, sequences packed from several documents): when
 * doc_start is given ([B][T_new], the position of the first token of the
 * document holding token i), the row reads only cached slots at or after that
 * position; the learned dummy slot stays visible to every row. Values outside
 * [0, position] are clamped into it. */
void wmo_channel_attend_doc(const wmo_dims *dm, const wmo_params *P, const double *Q,
                            const int *map, const int *ctx_len, const int *doc_start,
                            const double *Kc, const double *Vc, const int *rows, int nrows,
                            double *O)
{
    int B = dm->B, T = dm->T_new, L = dm->L, Hq = dm->Hq, Hkv = dm->Hkv, d = dm->d;
    int grp = Hq / Hkv;
    int cnt = list_len(rows, nrows, L * B * T);
#pragma omp parallel for schedule(dynamic)
    for (int t = 0; t < cnt; ++t) {
        int r = rows ? rows[t] : t;
        int l = r / (B * T), b = (r / T) % B, i = r % T;
        int c = map[l];
        long pos = (long)(ctx_len ? ctx_len[b] : 0) + i;
        int paper = dm->mask_mode == WMO_MASK_PAPER;
        long nvis = paper ? pos : pos + 1;  /* slots 0 .. nvis-1 before the document mask */
        long lo = doc_start ? doc_start[(size_t)b * T + i] : 0;
        if (lo < 0)
            lo = 0;
        if (lo > pos)
            lo = pos;
        for (int hh = 0; hh < Hq; ++hh) {
            int kvh = hh / grp;
            size_t base = (((size_t)c * B + b) * Hkv + kvh) * dm->S_cap * d + (size_t)lo * d;
            const double *q = Q + ((((size_t)l * B + b) * Hq + hh) * T + i) * d;
            const double *kd = paper ? P->Kd + ((size_t)c * Hkv + kvh) * d : NULL;
            const double *vd = paper ? P->Vd + ((size_t)c * Hkv + kvh) * d : NULL;
            wmo_attend_row(d, q, Kc + base, d, Vc + base, d, nvis - lo, kd, vd,
                           O + (((size_t)l * B + b) * T + i) * Hq * d + (size_t)hh * d);
        }
    }
}

void wmo_channel_attend(const wmo_dims *dm, const wmo_params *P, const double *Q, const int *map,
                        const int *ctx_len, const double *Kc, const double *Vc, const int *rows,
                        int nrows, double *O)
{
    wmo_channel_attend_doc(dm, P, Q, map, ctx_len, NULL, Kc, Vc, rows, nrows, O);
}

/* The fused step: pool the T_new new tokens into their slots, project the
 * consumer queries, then every consumer attends its channel. Slots below
 * ctx_len[b] must already hold the cached context. */
void wmo_layer_step_doc(const wmo_dims *dm, const wmo_params *P, const double *H, const int *map,
                        const int *ctx_len, const int *doc_start, double *Kc, double *Vc,
                        double *O)
{
    size_t nq = (size_t)dm->L * dm->B * dm->Hq * dm->T_new * dm->d;
    double *Q = (double *)malloc(sizeof(double) * nq);
    wmo_pool(dm, P, H, ctx_len, NULL, 0, Kc, Vc);
    wmo_q_project(dm, P, H, ctx_len, NULL, 0, Q);
    wmo_channel_attend_doc(dm, P, Q, map, ctx_len, doc_start, Kc, Vc, NULL, 0, O);
    free(Q);
}

void wmo_layer_step(const wmo_dims *dm, const wmo_params *P, const double *H, const int *map,
                    const int *ctx_len, double *Kc, double *Vc, double *O)
{
    wmo_layer_step_doc(dm, P, H, map, ctx_len, NULL, Kc, Vc, O);
}

int wmo_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ======================================= Section 3.3: the fixed-point passes
 *
 * The paper writes the exact solution as P = Pool(H), H = States(X; P): Pool
 * is Steps 1-2 applied at every position, States the decoder stack applied at
 * every position with each layer reading its channel of P. Here sequences
 * start empty (positions 0 .. T-1, one document per sequence), T = T_new and
 * S_cap >= T. Layouts: X[B][T][D] (the state entering layer 0 of each token,
 * i.e. its embedding), H[B][T][L][D] (states entering every layer), h_top[B][T][D]
 * (the state leaving the top layer), W_o[L][D][Hq*d].
 *
 * States needs the rest of each decoder block, which the method leaves
 * unchanged. A stand-in stands for it: h_{l+1} = h_l + W_o[l] o_l, the output
 * projection and residual of the attention sublayer, with o_l layer l's channel
 * attention (query from h_l, Qwen3 query side) and no MLP.
 */

/* The stand-in block: h_next = h_l + W_o[l] o_l, o_l of length Hq*d. */
void wmo_block_residual(const wmo_dims *dm, const double *W_o, int l, const double *h_l,
                        const double *o_l, double *h_next)
{
    int D = dm->D, HD = dm->Hq * dm->d;
    const double *W = W_o + (size_t)l * D * HD;
    for (int e = 0; e < D; ++e) {
        double a = 0.0;
        for (int c = 0; c < HD; ++c)
            a += W[(size_t)e * HD + c] * o_l[c];
        h_next[e] = h_l[e] + a;
    }
}

/* States at position i of sequence b: layers 0 .. L-1 in depth order, each
 * attending channel map[l] over the cache as it stands (dummy + slots < i, or
 * slots <= i in the inclusive mask). Writes the L states entering the layers to
 * Hrow[L][D] and the state leaving the top layer to top[D]. */
static void states_position(const wmo_dims *dm, const wmo_params *P, const double *W_o,
                            const int *map, const double *x, int b, int i, const double *Kc,
                            const double *Vc, double *Hrow, double *top)
{
    int L = dm->L, D = dm->D, Hq = dm->Hq, Hkv = dm->Hkv, d = dm->d, grp = Hq / Hkv;
    int paper = dm->mask_mode == WMO_MASK_PAPER;
    long nvis = paper ? i : i + 1;
    double *q = (double *)malloc(sizeof(double) * Hq * d);
    double *o = (double *)malloc(sizeof(double) * Hq * d);
    memcpy(Hrow, x, sizeof(double) * D);
    for (int l = 0; l < L; ++l) {
        const double *h = Hrow + (size_t)l * D;
        double *next = l + 1 < L ? Hrow + (size_t)(l + 1) * D : top;
        int c = map[l];
        wmo_query_token(dm, P, h, l, (double)i, q);
        for (int hh = 0; hh < Hq; ++hh) {
            int kvh = hh / grp;
            size_t base = (((size_t)c * dm->B + b) * Hkv + kvh) * dm->S_cap * d;
            const double *kd = paper ? P->Kd + ((size_t)c * Hkv + kvh) * d : NULL;
            const double *vd = paper ? P->Vd + ((size_t)c * Hkv + kvh) * d : NULL;
            wmo_attend_row(d, q + (size_t)hh * d, Kc + base, d, Vc + base, d, nvis, kd, vd,
                           o + (size_t)hh * d);
        }
        wmo_block_residual(dm, W_o, l, h, o, next);
    }
    free(o);
    free(q);
}

/* Pool at position i of sequence b (Steps 1-2): its L states -> cache slot i. */
static void pool_position(const wmo_dims *dm, const wmo_params *P, const double *Hrow, int b,
                          int i, double *Kc, double *Vc)
{
    int L = dm->L, k = dm->k, D = dm->D, KV = dm->k * dm->Hkv * dm->d;
    double *al = (double *)malloc(sizeof(double) * 2 * k * L);
    double *mx = (double *)malloc(sizeof(double) * 2 * k * D);
    double *kt = (double *)malloc(sizeof(double) * KV);
    double *vt = (double *)malloc(sizeof(double) * KV);
    wmo_pool_mix_token(dm, P, Hrow, al, mx);
    wmo_project_token(dm, P, mx, (double)i, kt, vt);
    store_cache_rows(dm, b, i, kt, vt, Kc, Vc);
    free(vt);
    free(kt);
    free(mx);
    free(al);
}

/* H^(0): every layer's state is the token's embedding. */
static void initial_states(const wmo_dims *dm, const double *X, double *H)
{
    int B = dm->B, T = dm->T_new, L = dm->L, D = dm->D;
    for (int b = 0; b < B; ++b)
        for (int i = 0; i < T; ++i)
            for (int l = 0; l < L; ++l)
                memcpy(H + (((size_t)b * T + i) * L + l) * D, X + ((size_t)b * T + i) * D,
                       sizeof(double) * D);
}

/* Jacobi iteration, Section 3.3: H^(0) = embeddings; for t = 1 .. passes,
 * P^(t) = Pool(H^(t-1)) at every position, then H^(t) = States(X; P^(t)) at
 * every position. Returns H^(passes), its top states, and the cache P^(passes). */
void wmo_jacobi(const wmo_dims *dm, const wmo_params *P, const double *W_o, const int *map,
                const double *X, int passes, double *H, double *h_top, double *Kc, double *Vc)
{
    int B = dm->B, T = dm->T_new, L = dm->L, D = dm->D;
    initial_states(dm, X, H);
    for (int t = 1; t <= passes; ++t) {
#pragma omp parallel for schedule(dynamic)
        for (int n = 0; n < B * T; ++n)
            pool_position(dm, P, H + (size_t)n * L * D, n / T, n % T, Kc, Vc);
#pragma omp parallel for schedule(dynamic)
        for (int n = 0; n < B * T; ++n)
            states_position(dm, P, W_o, map, X + (size_t)n * D, n / T, n % T, Kc, Vc,
                            H + (size_t)n * L * D, h_top + (size_t)n * D);
    }
}

/* Cyclic Gauss-Seidel iteration, Section 3.3: the positions split into g
 * strided groups G_q = {i : i mod g = q}. The cache starts as Pool(H^(0)); each
 * pass evaluates G_0 .. G_{g-1} in order, and group q first recomputes the
 * states of all its positions from the cache as it stands (so it reads the
 * current pass's updates of groups < q and the previous pass's of the rest,
 * its own included: a parallel Jacobi update within the group), then pools
 * them into its slots. g = 1 reproduces Jacobi iteration (its cache ends one
 * pool later: Pool(H^(passes))); g = T is autoregressive decoding. */
void wmo_gauss_seidel(const wmo_dims *dm, const wmo_params *P, const double *W_o,
                      const int *map, const double *X, int g, int passes, double *H,
                      double *h_top, double *Kc, double *Vc)
{
    int B = dm->B, T = dm->T_new, L = dm->L, D = dm->D;
    initial_states(dm, X, H);
#pragma omp parallel for schedule(dynamic)
    for (int n = 0; n < B * T; ++n)
        pool_position(dm, P, H + (size_t)n * L * D, n / T, n % T, Kc, Vc);
    for (int t = 1; t <= passes; ++t) {
        for (int q = 0; q < g; ++q) {
            int per = (T - q + g - 1) / g; /* positions q, q + g, ... below T */
#pragma omp parallel for schedule(dynamic)
            for (int u = 0; u < B * per; ++u) {
                int b = u / per, i = q + g * (u % per);
                size_t n = (size_t)b * T + i;
                states_position(dm, P, W_o, map, X + n * D, b, i, Kc, Vc, H + n * L * D,
                                h_top + n * D);
            }
#pragma omp parallel for schedule(dynamic)
            for (int u = 0; u < B * per; ++u) {
                int b = u / per, i = q + g * (u % per);
                pool_position(dm, P, H + ((size_t)b * T + i) * L * D, b, i, Kc, Vc);
            }
        }
    }
}

/* The same iteration from a given cache Kc0, Vc0 in place of Pool(H^(0)): the passes that
 * follow a point where the cache is held fixed, as in truncated backpropagation through
 * the last passes (Section 3.3). */
void wmo_gauss_seidel_from(const wmo_dims *dm, const wmo_params *P, const double *W_o,
                           const int *map, const double *X, int g, const double *Kc0,
                           const double *Vc0, int passes, double *H, double *h_top,
                           double *Kc, double *Vc)
{
    int B = dm->B, T = dm->T_new, L = dm->L, D = dm->D;
    size_t cache = (size_t)dm->k * B * dm->Hkv * dm->S_cap * dm->d;
    memcpy(Kc, Kc0, sizeof(double) * cache);
    memcpy(Vc, Vc0, sizeof(double) * cache);
    initial_states(dm, X, H);
    for (int t = 1; t <= passes; ++t) {
        for (int q = 0; q < g; ++q) {
            int per = (T - q + g - 1) / g;
#pragma omp parallel for schedule(dynamic)
            for (int u = 0; u < B * per; ++u) {
                int b = u / per, i = q + g * (u % per);
                size_t n = (size_t)b * T + i;
                states_position(dm, P, W_o, map, X + n * D, b, i, Kc, Vc, H + n * L * D,
                                h_top + n * D);
            }
#pragma omp parallel for schedule(dynamic)
            for (int u = 0; u < B * per; ++u) {
                int b = u / per, i = q + g * (u % per);
                pool_position(dm, P, H + ((size_t)b * T + i) * L * D, b, i, Kc, Vc);
            }
        }
    }
}

/* Exact left-to-right evaluation (Section 3.2): position by position, all L
 * layers in depth order against the cache of the earlier positions, then one
 * pool evaluation appends the position's channels. Defined in the paper's mask
 * only: with the inclusive mask a position would read its own slot before its
 * pool writes it. */
void wmo_autoregressive(const wmo_dims *dm, const wmo_params *P, const double *W_o,
                        const int *map, const double *X, double *H, double *h_top, double *Kc,
                        double *Vc)
{
    int B = dm->B, T = dm->T_new, L = dm->L, D = dm->D;
    for (int i = 0; i < T; ++i) {
#pragma omp parallel for schedule(dynamic)
        for (int b = 0; b < B; ++b) {
            size_t n = (size_t)b * T + i;
            states_position(dm, P, W_o, map, X + n * D, b, i, Kc, Vc, H + n * L * D,
                            h_top + n * D);
            pool_position(dm, P, H + n * L * D, b, i, Kc, Vc);
        }
    }
}

/* ============================ Section 3.1 Step 3: the dense soft read (variant)
 *
 * The paper contrasts its fixed one-channel selection with a dense read over all
 * channels that would permit learned soft assignments (and would stream all k
 * channels per layer). Read here as: layer l attends a soft mix of the channels,
 * K^_l[s] = sum_c w[l][c] K~_c[s], V^_l[s] = sum_c w[l][c] V_c[s], and likewise
 * for the dummy slot, with w[L][k] the layer's assignment weights as given (the
 * fixed selection is the one-hot row w[l][c] = [c == map[l]]). The attention is
 * then the standard one over the mixed slots. */
void wmo_channel_attend_dense(const wmo_dims *dm, const wmo_params *P, const double *w,
                              const double *Q, const int *ctx_len, const double *Kc,
                              const double *Vc, const int *rows, int nrows, double *O)
{
    int B = dm->B, T = dm->T_new, L = dm->L, k = dm->k, Hq = dm->Hq, Hkv = dm->Hkv, d = dm->d;
    int grp = Hq / Hkv;
    int cnt = list_len(rows, nrows, L * B * T);
#pragma omp parallel for schedule(dynamic)
    for (int t = 0; t < cnt; ++t) {
        int r = rows ? rows[t] : t;
        int l = r / (B * T), b = (r / T) % B, i = r % T;
        long pos = (long)(ctx_len ? ctx_len[b] : 0) + i;
        int paper = dm->mask_mode == WMO_MASK_PAPER;
        long nvis = paper ? pos : pos + 1;
        double *Km = (double *)malloc(sizeof(double) * (nvis > 0 ? nvis : 1) * d);
        double *Vm = (double *)malloc(sizeof(double) * (nvis > 0 ? nvis : 1) * d);
        double *kd = (double *)malloc(sizeof(double) * d);
        double *vd = (double *)malloc(sizeof(double) * d);
        for (int hh = 0; hh < Hq; ++hh) {
            int kvh = hh / grp;
            for (long s = 0; s < nvis; ++s)
                for (int e = 0; e < d; ++e) {
                    double a = 0.0, v = 0.0;
                    for (int c = 0; c < k; ++c) {
                        size_t off = ((((size_t)c * B + b) * Hkv + kvh) * dm->S_cap + s) * d + e;
                        a += w[(size_t)l * k + c] * Kc[off];
                        v += w[(size_t)l * k + c] * Vc[off];
                    }
                    Km[s * d + e] = a;
                    Vm[s * d + e] = v;
                }
            for (int e = 0; e < d; ++e) {
                double a = 0.0, v = 0.0;
                for (int c = 0; c < k; ++c) {
                    a += w[(size_t)l * k + c] * P->Kd[((size_t)c * Hkv + kvh) * d + e];
                    v += w[(size_t)l * k + c] * P->Vd[((size_t)c * Hkv + kvh) * d + e];
                }
                kd[e] = a;
                vd[e] = v;
            }
            const double *q = Q + ((((size_t)l * B + b) * Hq + hh) * T + i) * d;
            wmo_attend_row(d, q, Km, d, Vm, d, nvis, paper ? kd : NULL, paper ? vd : NULL,
                           O + (((size_t)l * B + b) * T + i) * Hq * d + (size_t)hh * d);
        }
        free(vd);
        free(kd);
        free(Vm);
        free(Km);
    }
}
