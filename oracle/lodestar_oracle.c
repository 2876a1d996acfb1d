/*
 * CPU oracle for the batched routing scorer -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct implementations of what the routing hot path
 * computes, written from the paper (Lodestar, arXiv 2606.00946).  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load this
 * library; the product path never does.  It shares no code, header, table or
 * helper with the HIP library.
 *
 * Precision modes:
 *   LSO_F64  -- the definition, evaluated in double precision.
 *   LSO_F32  -- the kernel's precision: fp32 values, every dot product an
 *               fmaf chain that starts from the bias and runs over the inputs in
 *               ascending order, no other contraction.
 *   LSO_BF16 -- as LSO_F32, but every layer's weights and input activations are
 *               first rounded to bfloat16 (round to nearest, ties to even).
 * Routing decisions are compared in the kernel's precision; scores are also
 * compared with the LSO_F64 definition within a tolerance.
 *
 * Build: gcc -O2 -mfma -ffp-contract=off -fopenmp -shared -fPIC
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { LSO_F64 = 0, LSO_F32 = 1, LSO_BF16 = 2 };
#define LSO_BLOCK_TOKENS 16
#define LSO_DERIVED 5
#define LSO_MAX_LAYERS 8

/* ------------------------------------------------------------------------- */
/* bfloat16 rounding from the number format's definition: 8 significant bits,  */
/* the same exponent range as binary32, round to nearest with ties to even.    */
/* ------------------------------------------------------------------------- */
float lso_bf16_round(float x)
{
    if (x == 0.0f || isinf(x)) return x;
    if (isnan(x)) return x;
    int e;
    double m = frexp((double)x, &e);           /* x = m * 2^e, 0.5 <= |m| < 1 */
    (void)m;
    if (e < -125) e = -125;                    /* below binary32's smallest normal the quantum stays 2^-133 */
    double scale = ldexp(1.0, 8 - e);          /* 8 significant bits */
    double q = nearbyint((double)x * scale);   /* ties-to-even in the default rounding mode */
    double r = q / scale;
    if (fabs(r) >= ldexp(1.0, 128)) return (float)copysign(INFINITY, r);
    return (float)r;
}

/* ------------------------------------------------------------------------- */
/* Prefix overlap (Section 2 Background: prefix reuse is strictly sequential,  */
/* a cached block helps only if every earlier block is cached too; Section    */
/* 4.2 Prefix KV cache tracker: tokenized prompt in, per-instance hit out).    */
/* The overlap of request r on instance i is the number of leading blocks of   */
/* r that are all in instance i's cached set.                                  */
/* ------------------------------------------------------------------------- */
static int cmp_u64(const void* a, const void* b)
{
    uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
    return (x > y) - (x < y);
}

typedef struct { uint64_t* keys; int64_t count; } lso_set;

static void build_sets(int32_t N, const int64_t* inst_off, const uint64_t* hashes, lso_set* sets)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t i = 0; i < N; ++i) {
        int64_t c = inst_off[i + 1] - inst_off[i];
        uint64_t* k = (uint64_t*)malloc((size_t)(c > 0 ? c : 1) * sizeof(uint64_t));
        memcpy(k, hashes + inst_off[i], (size_t)c * sizeof(uint64_t));
        qsort(k, (size_t)c, sizeof(uint64_t), cmp_u64);
        int64_t u = 0;                          /* order and duplicates are irrelevant to a set */
        for (int64_t t = 0; t < c; ++t)
            if (u == 0 || k[u - 1] != k[t]) k[u++] = k[t];
        sets[i].keys = k;
        sets[i].count = u;
    }
}

static void free_sets(int32_t N, lso_set* sets)
{
    for (int32_t i = 0; i < N; ++i) free(sets[i].keys);
}

static int in_set(const lso_set* s, uint64_t key)
{
    return bsearch(&key, s->keys, (size_t)s->count, sizeof(uint64_t), cmp_u64) != NULL;
}

static int32_t overlap_one(const uint64_t* h, int64_t n, const lso_set* s)
{
    int32_t l = 0;
    for (int64_t j = 0; j < n; ++j) {
        if (!in_set(s, h[j])) break;
        ++l;
    }
    return l;
}

static void set_threads(int threads)
{
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#else
    (void)threads;
#endif
}

/* out[q*N + i] = overlap of request sel[q] (all requests when sel == NULL) on instance i */
int lso_overlap(int32_t n_sel, const int32_t* sel, const int64_t* req_off, const uint64_t* req_hashes,
                int32_t N, const int64_t* inst_off, const uint64_t* inst_hashes, int32_t* out, int threads)
{
    set_threads(threads);
    lso_set* sets = (lso_set*)calloc((size_t)N, sizeof(lso_set));
    if (!sets) return -2;
    build_sets(N, inst_off, inst_hashes, sets);
#pragma omp parallel for schedule(dynamic, 4)
    for (int32_t q = 0; q < n_sel; ++q) {
        int32_t r = sel ? sel[q] : q;
        for (int32_t i = 0; i < N; ++i)
            out[(int64_t)q * N + i] = overlap_one(req_hashes + req_off[r], req_off[r + 1] - req_off[r], &sets[i]);
    }
    free_sets(N, sets);
    free(sets);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Pair features (Section 4.1, Features; Alg. 4 inputs).  The raw row is the   */
/* instance state followed by the request and pair columns:                    */
/*   [ inst_feat[i] | L, n | l, kappa, u ]                                     */
/* L = prompt tokens, n = hashed blocks, l = overlap in blocks,                */
/* kappa = 16 l / L the expected hit ratio (Section 2: fraction of the input   */
/* tokens whose KV blocks are already cached; 0 when L = 0), u = L - 16 l the  */
/* tokens left to prefill.  kappa is divided in the mode's precision.          */
/* ------------------------------------------------------------------------- */
void lso_features(int mode, int32_t d_inst, const float* inst_row, int32_t L, int32_t n, int32_t l, double* x)
{
    for (int32_t c = 0; c < d_inst; ++c) x[c] = (double)inst_row[c];
    x[d_inst + 0] = (double)L;
    x[d_inst + 1] = (double)n;
    x[d_inst + 2] = (double)l;
    int64_t hit_tokens = (int64_t)LSO_BLOCK_TOKENS * l;
    if (L == 0) x[d_inst + 3] = 0.0;
    else if (mode == LSO_F64) x[d_inst + 3] = (double)hit_tokens / (double)L;
    else x[d_inst + 3] = (double)((float)hit_tokens / (float)L);
    x[d_inst + 4] = (double)((int64_t)L - hit_tokens);
}

/* ------------------------------------------------------------------------- */
/* Reward model (Section 4.1, Request-instance reward model / Model            */
/* architecture): one MLP shared by every instance, ReLU hidden layers, scalar */
/* output.  The output is the predicted TTFT in seconds; the reward is its     */
/* negation.  Inputs are z-scored per feature first (Alg. 4, Normalize).       */
/* Parameters are packed per layer as W [out x in] row-major, then b [out].    */
/* ------------------------------------------------------------------------- */
typedef struct {
    int n_layers;
    int in[LSO_MAX_LAYERS], out[LSO_MAX_LAYERS];
    const float* W[LSO_MAX_LAYERS];
    const float* b[LSO_MAX_LAYERS];
    int64_t W_off[LSO_MAX_LAYERS], b_off[LSO_MAX_LAYERS];
    int max_width;
} lso_net;

static int net_init(lso_net* net, int32_t d, int32_t n_hidden, const int32_t* hidden, const float* params)
{
    if (n_hidden < 0 || n_hidden + 1 > LSO_MAX_LAYERS || d < 1) return -1;
    int64_t off = 0;
    int prev = d;
    net->n_layers = n_hidden + 1;
    net->max_width = d;
    for (int l = 0; l < net->n_layers; ++l) {
        int o = (l < n_hidden) ? hidden[l] : 1;
        if (o < 1) return -1;
        net->in[l] = prev;
        net->out[l] = o;
        net->W_off[l] = off;
        net->W[l] = params ? params + off : NULL;
        off += (int64_t)o * prev;
        net->b_off[l] = off;
        net->b[l] = params ? params + off : NULL;
        off += o;
        if (o > net->max_width) net->max_width = o;
        prev = o;
    }
    return 0;
}

int64_t lso_param_count(int32_t d, int32_t n_hidden, const int32_t* hidden)
{
    lso_net net;
    if (net_init(&net, d, n_hidden, hidden, NULL)) return -1;
    int l = net.n_layers - 1;
    return net.b_off[l] + net.out[l];
}

/* One pair, definition in double precision. */
static double forward_f64(const lso_net* net, const float* mu, const float* inv_sigma, const double* x,
                          double* buf_a, double* buf_b)
{
    int d = net->in[0];
    for (int k = 0; k < d; ++k) buf_a[k] = (x[k] - (double)mu[k]) * (double)inv_sigma[k];
    double* a = buf_a;
    double* z = buf_b;
    for (int l = 0; l < net->n_layers; ++l) {
        int K = net->in[l], O = net->out[l];
        for (int j = 0; j < O; ++j) {
            double acc = (double)net->b[l][j];
            for (int k = 0; k < K; ++k) acc += (double)net->W[l][(int64_t)j * K + k] * a[k];
            z[j] = acc;
        }
        if (l + 1 == net->n_layers) return z[0];
        for (int j = 0; j < O; ++j) z[j] = z[j] > 0.0 ? z[j] : 0.0;
        double* t = a; a = z; z = t;
    }
    return 0.0;
}

/* Copy of the parameters with every weight (not bias) rounded to bf16. */
static float* bf16_weights(const lso_net* net, const float* params)
{
    int l = net->n_layers - 1;
    int64_t P = net->b_off[l] + net->out[l];
    float* q = (float*)malloc(sizeof(float) * (size_t)P);
    memcpy(q, params, sizeof(float) * (size_t)P);
    for (l = 0; l < net->n_layers; ++l)
        for (int64_t t = 0; t < (int64_t)net->out[l] * net->in[l]; ++t)
            q[net->W_off[l] + t] = lso_bf16_round(params[net->W_off[l] + t]);
    return q;
}

/* One pair in the kernel's precision (fp32 fma chains, optional bf16 operands).
 * In LSO_BF16 mode `net` must already hold bf16-rounded weights (bf16_weights);
 * the inputs and activations of every layer are rounded here.  `last`
 * (nullable) receives the input of the output layer (the last hidden layer's
 * activations). */
static float forward_lowp(int mode, const lso_net* net, const float* mu, const float* inv_sigma, const double* x,
                          float* buf_a, float* buf_b, float* last)
{
    int bf = (mode == LSO_BF16);
    int d = net->in[0];
    for (int k = 0; k < d; ++k) {
        float xf = (float)x[k];
        float t = xf - mu[k];
        t = t * inv_sigma[k];
        buf_a[k] = bf ? lso_bf16_round(t) : t;
    }
    float* a = buf_a;
    float* z = buf_b;
    for (int l = 0; l < net->n_layers; ++l) {
        int K = net->in[l], O = net->out[l];
        for (int j = 0; j < O; ++j) {
            float acc = net->b[l][j];
            for (int k = 0; k < K; ++k) {
                acc = fmaf(net->W[l][(int64_t)j * K + k], a[k], acc);
            }
            z[j] = acc;
        }
        if (l + 1 == net->n_layers) {
            if (last) memcpy(last, a, sizeof(float) * (size_t)K);
            return z[0];
        }
        for (int j = 0; j < O; ++j) {
            float h = z[j] > 0.0f ? z[j] : 0.0f;
            z[j] = bf ? lso_bf16_round(h) : h;
        }
        float* t = a; a = z; z = t;
    }
    return 0.0f;
}

/* scores[r] for raw feature rows x [rows x d] (double holding the raw values). */
int lso_forward(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, const float* params,
                const float* mu, const float* inv_sigma, int64_t rows, const double* x, double* scores, int threads)
{
    lso_net net;
    if (net_init(&net, d, n_hidden, hidden, params)) return -1;
    float* q = NULL;
    if (mode == LSO_BF16) {
        q = bf16_weights(&net, params);
        net_init(&net, d, n_hidden, hidden, q);
    }
    set_threads(threads);
#pragma omp parallel
    {
        double* da = (double*)malloc(sizeof(double) * (size_t)net.max_width);
        double* db = (double*)malloc(sizeof(double) * (size_t)net.max_width);
        float* fa = (float*)malloc(sizeof(float) * (size_t)net.max_width);
        float* fb = (float*)malloc(sizeof(float) * (size_t)net.max_width);
#pragma omp for schedule(static)
        for (int64_t r = 0; r < rows; ++r) {
            const double* xr = x + r * d;
            scores[r] = (mode == LSO_F64) ? forward_f64(&net, mu, inv_sigma, xr, da, db)
                                          : (double)forward_lowp(mode, &net, mu, inv_sigma, xr, fa, fb, NULL);
        }
        free(da); free(db); free(fa); free(fb);
    }
    free(q);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Greedy routing (Section 4.1: route to the highest predicted reward; Alg. 4  */
/* argmax).  With the model predicting TTFT this is the smallest prediction.   */
/* Ties go to the lowest instance id; -0 equals +0; NaN ranks after +inf, so   */
/* NaN wins only when every score is NaN, and then instance 0 wins.            */
/* ------------------------------------------------------------------------- */
static int better(double a, int32_t ia, double b, int32_t ib)
{
    if (isnan(a)) return isnan(b) && ia < ib;
    if (isnan(b)) return 1;
    if (a < b) return 1;
    if (a > b) return 0;
    return ia < ib;
}

int32_t lso_argmin(int32_t N, const double* scores, double* min_out)
{
    int32_t best = 0;
    for (int32_t i = 1; i < N; ++i)
        if (better(scores[i], i, scores[best], best)) best = i;
    if (min_out) *min_out = N > 0 ? scores[best] : NAN;
    return best;
}

/* ------------------------------------------------------------------------- */
/* Whole scoring pass for selected requests: overlap, features, model, argmin. */
/* Outputs are indexed by position q in sel (all requests when sel == NULL).   */
/* feat_out (nullable) receives the raw feature row of the chosen pair.        */
/* ------------------------------------------------------------------------- */
int lso_score(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, const float* params,
              const float* mu, const float* inv_sigma,
              int32_t n_sel, const int32_t* sel, const int64_t* req_off, const uint64_t* req_hashes,
              const int32_t* prompt_len, int32_t N, const float* inst_feat,
              const int64_t* inst_off, const uint64_t* inst_hashes,
              int32_t* overlap_out, double* scores_out, int32_t* chosen_out, double* min_out,
              double* feat_out, int threads)
{
    lso_net net;
    if (net_init(&net, d, n_hidden, hidden, params)) return -1;
    if (d <= LSO_DERIVED || N < 1) return -1;
    int32_t d_inst = d - LSO_DERIVED;
    float* q = NULL;
    if (mode == LSO_BF16) {
        q = bf16_weights(&net, params);
        net_init(&net, d, n_hidden, hidden, q);
    }
    set_threads(threads);
    lso_set* sets = (lso_set*)calloc((size_t)N, sizeof(lso_set));
    if (!sets) return -2;
    build_sets(N, inst_off, inst_hashes, sets);
#pragma omp parallel
    {
        double* x = (double*)malloc(sizeof(double) * (size_t)d * (size_t)N);
        double* s = (double*)malloc(sizeof(double) * (size_t)N);
        int32_t* ov = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
        double* da = (double*)malloc(sizeof(double) * (size_t)net.max_width);
        double* db = (double*)malloc(sizeof(double) * (size_t)net.max_width);
        float* fa = (float*)malloc(sizeof(float) * (size_t)net.max_width);
        float* fb = (float*)malloc(sizeof(float) * (size_t)net.max_width);
#pragma omp for schedule(dynamic, 1)
        for (int32_t q = 0; q < n_sel; ++q) {
            int32_t r = sel ? sel[q] : q;
            int64_t n = req_off[r + 1] - req_off[r];
            for (int32_t i = 0; i < N; ++i) {
                ov[i] = overlap_one(req_hashes + req_off[r], n, &sets[i]);
                double* xi = x + (int64_t)i * d;
                lso_features(mode, d_inst, inst_feat + (int64_t)i * d_inst, prompt_len[r], (int32_t)n, ov[i], xi);
                s[i] = (mode == LSO_F64) ? forward_f64(&net, mu, inv_sigma, xi, da, db)
                                         : (double)forward_lowp(mode, &net, mu, inv_sigma, xi, fa, fb, NULL);
            }
            double m;
            int32_t c = lso_argmin(N, s, &m);
            if (overlap_out) memcpy(overlap_out + (int64_t)q * N, ov, sizeof(int32_t) * (size_t)N);
            if (scores_out) memcpy(scores_out + (int64_t)q * N, s, sizeof(double) * (size_t)N);
            if (chosen_out) chosen_out[q] = c;
            if (min_out) min_out[q] = m;
            if (feat_out) memcpy(feat_out + (int64_t)q * d, x + (int64_t)c * d, sizeof(double) * (size_t)d);
        }
        free(x); free(s); free(ov); free(da); free(db); free(fa); free(fb);
    }
    free_sets(N, sets);
    free(sets);
    free(q);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Online update (Section 4.3.2: the predictor is retrained on recent          */
/* (features, observed TTFT) records).  The paper does not state the loss or   */
/* the optimiser; this is one plain SGD step on the mean squared error,        */
/*   L = (1/B) sum_b (t_b - y_b)^2,   W <- W - lr * dL/dW,                      */
/* with gradients by the chain rule through the ReLU layers and accumulated in */
/* double precision over samples in ascending order.                           */
/* LSO_F64 evaluates everything in double precision.  LSO_F32 and LSO_BF16    */
/* run the forward pass in the kernel's precision -- the same fp32 fma chains  */
/* as the scoring path -- so the ReLU masks, which floating point decides, are */
/* taken in that precision; the backward sums stay in double.  LSO_BF16 also   */
/* rounds to bfloat16 exactly the quantities the kernel holds in bfloat16      */
/* (inputs, weights and activations of every layer, and every layer's output   */
/* gradient before it multiplies anything); a gradient that is rounded is      */
/* itself summed in the kernel's precision, an fp32 chain in ascending order.  */
/* grad_out (nullable, double, same packing as params), loss_out (nullable).   */
/* ------------------------------------------------------------------------- */
uint64_t lso_splitmix64_mix(uint64_t z);

/* Dropout on the hidden activations while training (Section 4.1 Model         */
/* architecture: the predictor uses dropout 0.1).  Inverted dropout: a kept     */
/* unit is scaled by 1/(1-p) (in the kernel's precision, an fp32 multiply by    */
/* the fp32 value of 1/(1-p), before any bf16 rounding of the next layer's     */
/* input), a dropped one is 0; the backward pass multiplies the unit's          */
/* gradient by the same factor.  Unit j of hidden layer l for row b of update   */
/* call `step` draws the splitmix64 output number c + 1 for seed `seed`, with   */
/* c = ((step * 4 + l) * 2^24 + b) * 2^10 + j, and is dropped when the draw's   */
/* top 53 bits are below floor(p * 2^53).                                       */
static int lso_dropped(uint64_t seed, uint64_t step, int layer, int64_t row, int unit, uint64_t thr53)
{
    if (thr53 == 0) return 0;
    uint64_t c = ((((step * 4u + (uint64_t)layer) << 24) | (uint64_t)row) << 10) | (uint64_t)unit;
    uint64_t u = lso_splitmix64_mix(seed + (c + 1u) * 0x9e3779b97f4a7c15ull);
    return (u >> 11) < thr53;
}

/* One SGD step with dropout rate p in [0, 1) (p = 0: none); rows must be      */
/* fewer than 2^24, hidden widths at most 2^10, step below 2^36.               */
int lso_update_dropout(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, float* params,
                       const float* mu, const float* inv_sigma, int32_t B, const float* feats, const float* ttft,
                       float lr, double p, uint64_t seed, uint64_t step, double* grad_out, double* loss_out)
{
    lso_net net;
    if (net_init(&net, d, n_hidden, hidden, params)) return -1;
    if (B < 1) return -1;
    if (!(p >= 0.0 && p < 1.0) || B >= (1 << 24)) return -1;
    for (int l = 0; l < n_hidden; ++l)
        if (hidden[l] > 1024) return -1;
    int bf = (mode == LSO_BF16);
    int lowp = (mode == LSO_F32 || mode == LSO_BF16);
    int L = net.n_layers;
    uint64_t thr53 = (uint64_t)ldexp(p, 53);          /* dropped: top 53 bits below this */
    float scale_f = (float)(1.0 / (1.0 - p));         /* kernel precision */
    double scale_d = 1.0 / (1.0 - p);                 /* the definition */
    int64_t P = lso_param_count(d, n_hidden, hidden);
    double* grad = (double*)calloc((size_t)P, sizeof(double));
    int W = net.max_width;
    /* act[l] = input of layer l (act[0] = normalised features), pre[l] = pre-activation of layer l */
    double* act = (double*)malloc(sizeof(double) * (size_t)W * (size_t)(L + 1));
    double* pre = (double*)malloc(sizeof(double) * (size_t)W * (size_t)L);
    double* delta = (double*)malloc(sizeof(double) * (size_t)W);
    double* dnext = (double*)malloc(sizeof(double) * (size_t)W);
    /* weights as used by the arithmetic of this mode */
    double* Wq = (double*)malloc(sizeof(double) * (size_t)P);
    for (int64_t t = 0; t < P; ++t) Wq[t] = (double)params[t];
    if (bf)
        for (int l = 0; l < L; ++l)
            for (int64_t t = 0; t < (int64_t)net.out[l] * net.in[l]; ++t)
                Wq[net.W_off[l] + t] = (double)lso_bf16_round(params[net.W_off[l] + t]);
    double loss = 0.0;

    for (int32_t b = 0; b < B; ++b) {
        const float* xb = feats + (int64_t)b * d;
        double* a0 = act;
        for (int k = 0; k < d; ++k) {
            if (lowp) {
                float t = xb[k] - mu[k];
                t = t * inv_sigma[k];
                a0[k] = bf ? (double)lso_bf16_round(t) : (double)t;
            } else {
                a0[k] = ((double)xb[k] - (double)mu[k]) * (double)inv_sigma[k];
            }
        }
        /* forward */
        for (int l = 0; l < L; ++l) {
            int K = net.in[l], O = net.out[l];
            const double* a = act + (int64_t)l * W;
            double* z = pre + (int64_t)l * W;
            double* an = act + (int64_t)(l + 1) * W;
            for (int j = 0; j < O; ++j) {
                double acc;
                if (lowp) {
                    float f = params[net.b_off[l] + j];
                    for (int k = 0; k < K; ++k) f = fmaf((float)Wq[net.W_off[l] + (int64_t)j * K + k], (float)a[k], f);
                    acc = (double)f;
                } else {
                    acc = (double)params[net.b_off[l] + j];
                    for (int k = 0; k < K; ++k) acc += Wq[net.W_off[l] + (int64_t)j * K + k] * a[k];
                }
                z[j] = acc;
                if (l + 1 < L) {
                    double h = acc > 0.0 ? acc : 0.0;
                    if (lso_dropped(seed, step, l, b, j, thr53)) h = 0.0;
                    else if (thr53) h = lowp ? (double)((float)h * scale_f) : h * scale_d;
                    an[j] = bf ? (double)lso_bf16_round((float)h) : h;
                }
            }
        }
        double t_hat = pre[(int64_t)(L - 1) * W];
        double err = t_hat - (double)ttft[b];
        loss += err * err;
        /* backward: delta holds dL/dz of the current layer */
        double g = 2.0 * err / (double)B;
        delta[0] = bf ? (double)lso_bf16_round((float)g) : g;
        for (int l = L - 1; l >= 0; --l) {
            int K = net.in[l], O = net.out[l];
            const double* a = act + (int64_t)l * W;
            for (int j = 0; j < O; ++j) {
                double dj = delta[j];
                double* gw = grad + net.W_off[l] + (int64_t)j * K;
                for (int k = 0; k < K; ++k) gw[k] += dj * a[k];
                grad[net.b_off[l] + j] += dj;
            }
            if (l == 0) break;
            const double* zp = pre + (int64_t)(l - 1) * W;
            for (int k = 0; k < K; ++k) {
                double s = 0.0;
                if (bf) {
                    /* rounded to bf16 below, so summed in the kernel's precision:
                       an fp32 fma chain over the output units in ascending order */
                    float f = 0.0f;
                    for (int j = 0; j < O; ++j) f = fmaf((float)Wq[net.W_off[l] + (int64_t)j * K + k], (float)delta[j], f);
                    s = (double)f;
                } else {
                    for (int j = 0; j < O; ++j) s += Wq[net.W_off[l] + (int64_t)j * K + k] * delta[j];
                }
                double dk = zp[k] > 0.0 ? s : 0.0;
                if (lso_dropped(seed, step, l - 1, b, k, thr53)) dk = 0.0;
                else if (thr53) dk = bf ? (double)((float)dk * scale_f) : dk * (lowp ? (double)scale_f : scale_d);
                dnext[k] = bf ? (double)lso_bf16_round((float)dk) : dk;
            }
            memcpy(delta, dnext, sizeof(double) * (size_t)K);
        }
    }
    if (loss_out) *loss_out = loss / (double)B;
    for (int64_t t = 0; t < P; ++t) {
        if (grad_out) grad_out[t] = grad[t];
        params[t] = (float)((double)params[t] - (double)lr * grad[t]);
    }
    free(grad); free(act); free(pre); free(delta); free(dnext); free(Wq);
    return 0;
}

int lso_update(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, float* params,
               const float* mu, const float* inv_sigma, int32_t B, const float* feats, const float* ttft,
               float lr, double* grad_out, double* loss_out)
{
    return lso_update_dropout(mode, d, n_hidden, hidden, params, mu, inv_sigma, B, feats, ttft, lr, 0.0, 0, 0,
                              grad_out, loss_out);
}

/* ------------------------------------------------------------------------- */
/* Routing policy around the model: the gateway's routing with fallback       */
/* (Alg. 3), the routing service's logic (Alg. 4: cold start, out-of-range    */
/* guard, epsilon-greedy exploration, consistent-hashing K-filter, reward      */
/* tie-break) and the heuristic it falls back to (Alg. 1, or Alg. 2).          */
/* ------------------------------------------------------------------------- */

/* splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number     */
/* generators", 2014): the state advances by 0x9e3779b97f4a7c15 and each       */
/* output is the new state passed through this mixing function.                */
uint64_t lso_splitmix64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

/* Consistent hashing of a prefix group onto K instances (Section 4.1,        */
/* Consistent hashing based filtering), as rendezvous hashing: instance i's   */
/* weight for key k is output i+1 of splitmix64 seeded with k; the K heaviest */
/* instances (ties to the lower id) are selected, heaviest first.             */
int32_t lso_hrw_topk(int32_t N, uint64_t key, int32_t K, int32_t* out)
{
    int32_t n = K < N ? K : N;
    for (int32_t t = 0; t < n; ++t) {
        int32_t best = -1;
        uint64_t bw = 0;
        for (int32_t i = 0; i < N; ++i) {
            int taken = 0;
            for (int32_t u = 0; u < t; ++u) taken |= (out[u] == i);
            if (taken) continue;
            uint64_t w = lso_splitmix64_mix(key + 0x9e3779b97f4a7c15ull * (uint64_t)(i + 1));
            if (best < 0 || w > bw) { best = i; bw = w; }
        }
        out[t] = best;
    }
    return n;
}

static int32_t argmin_count(int32_t N, const double* c)
{
    int32_t b = 0;
    for (int32_t i = 1; i < N; ++i)
        if (c[i] < c[b]) b = i;
    return b;
}

/* Alg. 1 (prefix-cache-and-load) when alg == 1, Alg. 2 (prefix-aware with    */
/* threshold tau) when alg == 2.  m[i] is the prefix match ratio of the       */
/* request on instance i, c[i] its request count.  Mean and standard          */
/* deviation are the population ones, summed in ascending instance order.     */
/* Ties in every ordering go to the lower instance id.                        */
int32_t lso_heuristic(int32_t alg, int32_t N, const float* m, const double* c, double theta, double k, double tau)
{
    if (alg == 2) {
        int32_t b = 0;
        for (int32_t i = 1; i < N; ++i)
            if (m[i] > m[b]) b = i;
        if ((double)m[b] > tau) return b;
        return argmin_count(N, c);
    }
    double cmin = c[0], cmax = c[0];
    for (int32_t i = 1; i < N; ++i) {
        if (c[i] < cmin) cmin = c[i];
        if (c[i] > cmax) cmax = c[i];
    }
    if (cmax - cmin > theta) return argmin_count(N, c);
    double sum = 0.0;
    for (int32_t i = 0; i < N; ++i) sum += c[i];
    double mu = sum / (double)N;
    double var = 0.0;
    for (int32_t i = 0; i < N; ++i) var += (c[i] - mu) * (c[i] - mu);
    double sigma = sqrt(var / (double)N);
    double limit = mu + k * sigma;
    /* the first instance in (m desc, c asc, id asc) order that is not overloaded */
    int32_t b = -1;
    for (int32_t i = 0; i < N; ++i) {
        if (!(c[i] <= limit)) continue;
        if (b < 0 || m[i] > m[b] || (m[i] == m[b] && c[i] < c[b])) b = i;
    }
    return b >= 0 ? b : argmin_count(N, c);
}

typedef struct {
    int32_t heuristic;                  /* 1: Alg. 1, 2: Alg. 2 */
    int32_t count_col0, count_col1;     /* instance columns summed into the request count (-1: unused) */
    int32_t kv_col;                     /* instance column of KV-cache utilisation (-1: no K-filter) */
    int32_t k_filter;                   /* K (0: no K-filter) */
    int32_t pad;
    double theta_imbal, overload_k, prefix_tau;
    int64_t n_samples, n_min;
    double epsilon, tau_sat, tau_ben, delta;
    const float* lo;                    /* [d] feature bounds, NULL: no out-of-range guard */
    const float* hi;
} lso_policy;

#define LSO_ROUTE_OK 0
#define LSO_ROUTE_COLD_START 1
#define LSO_ROUTE_OOD 2
#define LSO_ROUTE_EXPLORED 0x100
#define LSO_ROUTE_KFILTER 0x200
#define LSO_ROUTE_TIEBREAK 0x400

static int in_bounds(float v, float lo, float hi) { return lo <= v && v <= hi; }

/* index of a 32-bit random word scaled onto [0, n) */
static int32_t scale_u32(uint32_t u, int64_t n) { return (int32_t)(((uint64_t)u * (uint64_t)n) >> 32); }

/* Routing decision for selected requests (outputs indexed by position in sel).
 * rnd holds three uniform 32-bit words per request (exploration draw,
 * exploration pick, tie-break pick), indexed by request id. */
int lso_route(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, const float* params,
              const float* mu, const float* inv_sigma,
              int32_t n_sel, const int32_t* sel, const int64_t* req_off, const uint64_t* req_hashes,
              const int32_t* prompt_len, int32_t N, const float* inst_feat,
              const int64_t* inst_off, const uint64_t* inst_hashes, const lso_policy* pol, const uint32_t* rnd,
              int32_t* chosen_out, int32_t* status_out, int32_t* heur_out, int threads)
{
    if (d <= LSO_DERIVED || N < 1) return -1;
    int32_t d_inst = d - LSO_DERIVED;
    int32_t Rsel = n_sel;
    int32_t* ov = (int32_t*)malloc(sizeof(int32_t) * (size_t)Rsel * N);
    double* sc = (double*)malloc(sizeof(double) * (size_t)Rsel * N);
    int rc = lso_score(mode, d, n_hidden, hidden, params, mu, inv_sigma, n_sel, sel, req_off, req_hashes, prompt_len,
                       N, inst_feat, inst_off, inst_hashes, ov, sc, NULL, NULL, NULL, threads);
    if (rc) { free(ov); free(sc); return rc; }
    /* per-instance quantities shared by every request */
    double* cnt = (double*)malloc(sizeof(double) * (size_t)N);
    int* inst_ok = (int*)malloc(sizeof(int) * (size_t)N);
    double kv_sum = 0.0;
    for (int32_t i = 0; i < N; ++i) {
        const float* row = inst_feat + (int64_t)i * d_inst;
        double ci = 0.0;
        if (pol->count_col0 >= 0) ci += (double)row[pol->count_col0];
        if (pol->count_col1 >= 0) ci += (double)row[pol->count_col1];
        cnt[i] = ci;
        int ok = 1;
        if (pol->lo)
            for (int32_t c = 0; c < d_inst; ++c) ok &= in_bounds(row[c], pol->lo[c], pol->hi[c]);
        inst_ok[i] = ok;
        if (pol->kv_col >= 0) kv_sum += (double)row[pol->kv_col];
    }
    int saturated = pol->kv_col >= 0 && kv_sum / (double)N > pol->tau_sat;
    uint64_t explore_thr = (uint64_t)floor(pol->epsilon * 4294967296.0);
    float* m = (float*)malloc(sizeof(float) * (size_t)N);
    int32_t* C = (int32_t*)malloc(sizeof(int32_t) * (size_t)(pol->k_filter > 0 ? pol->k_filter : 1));
    int32_t* S = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    for (int32_t q = 0; q < n_sel; ++q) {
        int32_t r = sel ? sel[q] : q;
        int64_t n = req_off[r + 1] - req_off[r];
        int32_t L = prompt_len[r];
        const double* s = sc + (int64_t)q * N;
        double kl_max = 0.0;
        for (int32_t i = 0; i < N; ++i) {
            /* the hit ratio as the feature row holds it, in the mode's precision */
            double row[LSO_DERIVED + 1];
            lso_features(mode, 0, NULL, L, (int32_t)n, ov[(int64_t)q * N + i], row);
            m[i] = (float)row[3];
            double kl = (double)m[i] * (double)L;
            if (i == 0 || kl > kl_max) kl_max = kl;
        }
        int32_t heur = lso_heuristic(pol->heuristic, N, m, cnt, pol->theta_imbal, pol->overload_k, pol->prefix_tau);
        int32_t chosen, status;
        int ood = 0;
        if (pol->lo) {
            ood |= !in_bounds((float)L, pol->lo[d_inst], pol->hi[d_inst]);
            ood |= !in_bounds((float)n, pol->lo[d_inst + 1], pol->hi[d_inst + 1]);
            for (int32_t i = 0; i < N; ++i) ood |= !inst_ok[i];
        }
        if (pol->n_samples < pol->n_min) {
            chosen = heur; status = LSO_ROUTE_COLD_START;
        } else if (ood) {
            chosen = heur; status = LSO_ROUTE_OOD;
        } else if ((uint64_t)rnd[(int64_t)r * 3] < explore_thr) {
            chosen = scale_u32(rnd[(int64_t)r * 3 + 1], N); status = LSO_ROUTE_OK | LSO_ROUTE_EXPLORED;
        } else {
            status = LSO_ROUTE_OK;
            chosen = lso_argmin(N, s, NULL);
            int32_t nc = 0;
            if (pol->k_filter > 0 && n >= 1 && saturated && kl_max > pol->tau_ben) {
                nc = lso_hrw_topk(N, req_hashes[req_off[r]], pol->k_filter, C);
                status |= LSO_ROUTE_KFILTER;
                int inC = 0;
                for (int32_t u = 0; u < nc; ++u) inC |= (C[u] == chosen);
                if (!inC) {
                    int32_t b = C[0];
                    for (int32_t u = 1; u < nc; ++u)
                        if (better(s[C[u]], C[u], s[b], b)) b = C[u];
                    chosen = b;
                }
            }
            double tb = s[chosen];
            if (pol->delta >= 0.0 && !isnan(tb)) {
                double lim = tb + pol->delta * fabs(tb);
                int32_t ns = 0;
                for (int32_t i = 0; i < N; ++i) {
                    int scope = 1;
                    if (nc > 0) {
                        scope = 0;
                        for (int32_t u = 0; u < nc; ++u) scope |= (C[u] == i);
                    }
                    if (scope && s[i] <= lim) S[ns++] = i;
                }
                if (ns > 1) {
                    chosen = S[scale_u32(rnd[(int64_t)r * 3 + 2], ns)];
                    status |= LSO_ROUTE_TIEBREAK;
                }
            }
        }
        if (chosen_out) chosen_out[q] = chosen;
        if (status_out) status_out[q] = status;
        if (heur_out) heur_out[q] = heur;
    }
    free(ov); free(sc); free(cnt); free(inst_ok); free(m); free(C); free(S);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Online-learning data path (Section 4.3.2, Training-data selection): a FIFO */
/* of the newest samples and a replay pool that admits samples evicted from  */
/* the FIFO by a gradient-coreset rule, and a retraining round over both.    */
/*                                                                           */
/* Gradient coreset: a sample's embedding is its prediction residual times   */
/* its last-hidden-layer activations, e = (t - y) a_L -- the gradient of the */
/* squared loss with respect to the output weights, up to the factor 2 --    */
/* evaluated with the current model in the kernel's precision (the residual  */
/* in fp32, the products and distances in double, summed over units in       */
/* ascending order).  Embeddings of the pool are re-evaluated at the start   */
/* of every push.  A candidate joins a pool with room; a full pool takes it  */
/* in place of its most redundant member (the one with the smallest nearest- */
/* neighbour distance, lowest slot on ties) when the candidate's distance to */
/* the pool is larger than that member's.  Candidates are the samples the    */
/* FIFO evicts, oldest first.                                                 */
/* ------------------------------------------------------------------------- */

static double emb_dist(const double* a, const double* b, int32_t H)
{
    double s = 0.0;
    for (int32_t j = 0; j < H; ++j) {
        double e = a[j] - b[j];
        s += e * e;
    }
    return s;
}

/* nearest neighbour of slot k among slots [0, n) other than k (lowest slot on ties) */
static void nn_of(const double* emb, int32_t H, int32_t n, int32_t k, double* dist, int32_t* idx)
{
    double best = INFINITY;
    int32_t bi = -1;
    for (int32_t j = 0; j < n; ++j) {
        if (j == k) continue;
        double v = emb_dist(emb + (int64_t)k * H, emb + (int64_t)j * H, H);
        if (v < best) { best = v; bi = j; }
    }
    *dist = best;
    *idx = bi;
}

/* Gradient-coreset embeddings of n raw rows: e[k][j] = (t_k - y_k) a_L[k][j]. */
int lso_embed(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, const float* params, const float* mu,
              const float* inv_sigma, int32_t n, const float* x, const float* y, double* emb)
{
    lso_net net;
    if (net_init(&net, d, n_hidden, hidden, params)) return -1;
    float* q = NULL;
    if (mode == LSO_BF16) {
        q = bf16_weights(&net, params);
        net_init(&net, d, n_hidden, hidden, q);
    }
    int32_t H = net.in[net.n_layers - 1];
    float* fa = (float*)malloc(sizeof(float) * (size_t)net.max_width);
    float* fb = (float*)malloc(sizeof(float) * (size_t)net.max_width);
    float* last = (float*)malloc(sizeof(float) * (size_t)H);
    double* xr = (double*)malloc(sizeof(double) * (size_t)d);
    for (int32_t k = 0; k < n; ++k) {
        for (int32_t c = 0; c < d; ++c) xr[c] = (double)x[(int64_t)k * d + c];
        float t = forward_lowp(mode == LSO_F64 ? LSO_F32 : mode, &net, mu, inv_sigma, xr, fa, fb, last);
        float res = t - y[k];
        for (int32_t j = 0; j < H; ++j) emb[(int64_t)k * H + j] = (double)res * (double)last[j];
    }
    free(fa); free(fb); free(last); free(xr); free(q);
    return 0;
}

int lso_buffer_push(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, const float* params,
                    const float* mu, const float* inv_sigma, int32_t fifo_cap, int32_t rep_cap,
                    int32_t* fifo_count, int32_t* fifo_head, float* fifo_x, float* fifo_y,
                    int32_t* rep_count, float* rep_x, float* rep_y, int32_t B, const float* x, const float* y,
                    int32_t* n_admitted)
{
    lso_net net;
    if (net_init(&net, d, n_hidden, hidden, params)) return -1;
    if (fifo_cap < 1 || rep_cap < 0 || B < 0) return -1;
    float* q = NULL;
    if (mode == LSO_BF16) {
        q = bf16_weights(&net, params);
        net_init(&net, d, n_hidden, hidden, q);
    }
    int32_t H = net.in[net.n_layers - 1];
    /* 1. the FIFO takes the new samples; the ones it evicts are the candidates, oldest first */
    float* cx = (float*)malloc(sizeof(float) * (size_t)(B > 0 ? B : 1) * d);
    float* cy = (float*)malloc(sizeof(float) * (size_t)(B > 0 ? B : 1));
    int32_t nc = 0;
    for (int32_t b = 0; b < B; ++b) {
        if (*fifo_count < fifo_cap) {
            int32_t slot = (*fifo_head + *fifo_count) % fifo_cap;
            memcpy(fifo_x + (int64_t)slot * d, x + (int64_t)b * d, sizeof(float) * (size_t)d);
            fifo_y[slot] = y[b];
            ++*fifo_count;
        } else {
            int32_t slot = *fifo_head;
            memcpy(cx + (int64_t)nc * d, fifo_x + (int64_t)slot * d, sizeof(float) * (size_t)d);
            cy[nc++] = fifo_y[slot];
            memcpy(fifo_x + (int64_t)slot * d, x + (int64_t)b * d, sizeof(float) * (size_t)d);
            fifo_y[slot] = y[b];
            *fifo_head = (slot + 1) % fifo_cap;
        }
    }
    /* 2. embeddings of the pool and of the candidates with the current model */
    int32_t n0 = *rep_count;
    double* emb = (double*)malloc(sizeof(double) * (size_t)(rep_cap > 0 ? rep_cap : 1) * H);
    double* ce = (double*)malloc(sizeof(double) * (size_t)(nc > 0 ? nc : 1) * H);
    if (n0 > 0) lso_embed(mode, d, n_hidden, hidden, params, mu, inv_sigma, n0, rep_x, rep_y, emb);
    if (nc > 0) lso_embed(mode, d, n_hidden, hidden, params, mu, inv_sigma, nc, cx, cy, ce);
    /* 3. nearest neighbours inside the pool */
    double* nnd = (double*)malloc(sizeof(double) * (size_t)(rep_cap > 0 ? rep_cap : 1));
    int32_t* nni = (int32_t*)malloc(sizeof(int32_t) * (size_t)(rep_cap > 0 ? rep_cap : 1));
    for (int32_t k = 0; k < n0; ++k) nn_of(emb, H, n0, k, &nnd[k], &nni[k]);
    /* 4. admission, one candidate at a time */
    int32_t n = n0, admitted = 0;
    for (int32_t c = 0; c < nc && rep_cap > 0; ++c) {
        const double* e = ce + (int64_t)c * H;
        int32_t slot;
        if (n < rep_cap) {
            slot = n++;
        } else {
            double dc = INFINITY;
            for (int32_t k = 0; k < n; ++k) {
                double v = emb_dist(e, emb + (int64_t)k * H, H);
                if (v < dc) dc = v;
            }
            int32_t js = 0;
            for (int32_t k = 1; k < n; ++k)
                if (nnd[k] < nnd[js]) js = k;
            if (!(dc > nnd[js])) continue;
            slot = js;
        }
        memcpy(emb + (int64_t)slot * H, e, sizeof(double) * (size_t)H);
        memcpy(rep_x + (int64_t)slot * d, cx + (int64_t)c * d, sizeof(float) * (size_t)d);
        rep_y[slot] = cy[c];
        ++admitted;
        for (int32_t k = 0; k < n; ++k) {
            if (k == slot) continue;
            if (nni[k] == slot) {
                nn_of(emb, H, n, k, &nnd[k], &nni[k]);
            } else {
                double v = emb_dist(emb + (int64_t)k * H, e, H);
                if (v < nnd[k] || (v == nnd[k] && slot < nni[k])) { nnd[k] = v; nni[k] = slot; }
            }
        }
        nn_of(emb, H, n, slot, &nnd[slot], &nni[slot]);
    }
    *rep_count = n;
    if (n_admitted) *n_admitted = admitted;
    free(cx); free(cy); free(emb); free(ce); free(nnd); free(nni); free(q);
    return 0;
}

/* One retraining round over the FIFO (oldest first) and the pool (by slot):  */
/* per epoch the samples are visited in the order perm gives (NULL: natural), */
/* in minibatches of `batch` (the last one may be shorter), one SGD step of   */
/* lso_update each.  loss_out (nullable) gets the mean minibatch loss of the  */
/* last epoch.                                                                 */
int lso_train_round_dropout(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, float* params,
                            const float* mu, const float* inv_sigma, int32_t fifo_cap, int32_t fifo_count,
                            int32_t fifo_head, const float* fifo_x, const float* fifo_y, int32_t rep_count,
                            const float* rep_x, const float* rep_y, int32_t epochs, int32_t batch, float lr,
                            const int32_t* perm, double p, uint64_t seed, uint64_t step0, double* loss_out)
{
    uint64_t step = step0;                       /* each minibatch is one update call */
    int32_t n = fifo_count + rep_count;
    if (n < 1 || batch < 1 || epochs < 0) return -1;
    float* X = (float*)malloc(sizeof(float) * (size_t)n * d);
    float* Y = (float*)malloc(sizeof(float) * (size_t)n);
    for (int32_t k = 0; k < fifo_count; ++k) {
        int32_t slot = (fifo_head + k) % fifo_cap;
        memcpy(X + (int64_t)k * d, fifo_x + (int64_t)slot * d, sizeof(float) * (size_t)d);
        Y[k] = fifo_y[slot];
    }
    for (int32_t k = 0; k < rep_count; ++k) {
        memcpy(X + (int64_t)(fifo_count + k) * d, rep_x + (int64_t)k * d, sizeof(float) * (size_t)d);
        Y[fifo_count + k] = rep_y[k];
    }
    float* bx = (float*)malloc(sizeof(float) * (size_t)batch * d);
    float* by = (float*)malloc(sizeof(float) * (size_t)batch);
    double last = 0.0;
    for (int32_t ep = 0; ep < epochs; ++ep) {
        double lsum = 0.0;
        int32_t nb = 0;
        for (int32_t s = 0; s < n; s += batch) {
            int32_t m = n - s < batch ? n - s : batch;
            for (int32_t u = 0; u < m; ++u) {
                int32_t k = perm ? perm[(int64_t)ep * n + s + u] : s + u;
                memcpy(bx + (int64_t)u * d, X + (int64_t)k * d, sizeof(float) * (size_t)d);
                by[u] = Y[k];
            }
            double loss;
            int rc = lso_update_dropout(mode, d, n_hidden, hidden, params, mu, inv_sigma, m, bx, by, lr, p, seed,
                                        step++, NULL, &loss);
            if (rc) { free(X); free(Y); free(bx); free(by); return rc; }
            lsum += loss;
            ++nb;
        }
        last = lsum / (double)nb;
    }
    if (loss_out) *loss_out = last;
    free(X); free(Y); free(bx); free(by);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Prefix-index maintenance (Section 2 Background: after routing a request the */
/* gateway records the request's prefix blocks on the chosen instance, and    */
/* each engine evicts its least recently used KV blocks; Section 4.2 Prefix   */
/* KV cache tracker: the index follows the gateway's own routing history).    */
/*                                                                             */
/* Every cached block carries a recency stamp, larger = more recent.  A commit */
/* of a routed batch (epoch e >= 1) touches, for each request r with a chosen  */
/* instance, each of its blocks k on that instance with stamp                  */
/*     e * 2^44 + r * 2^20 + (2^20 - 1 - k),                                   */
/* so later commits beat earlier ones, later requests of a batch beat earlier  */
/* ones, and within a request a block nearer the prompt's start is the more    */
/* recent (an engine frees a sequence's tail first, so what stays cached of a  */
/* request is a prefix of it).  A block keeps the largest stamp it was given.  */
/* Then every instance holding more than its capacity drops its smallest      */
/* stamps until it holds exactly its capacity.  Loaded state: entry j of an   */
/* instance's list has stamp j + 1 (list order = oldest first).               */
/* ------------------------------------------------------------------------- */
#define LSO_STAMP_K_BITS 20
#define LSO_STAMP_R_BITS 24
#define LSO_STAMP_E_BITS 20

uint64_t lso_stamp(uint32_t epoch, uint32_t r, uint32_t k)
{
    return ((uint64_t)epoch << (LSO_STAMP_K_BITS + LSO_STAMP_R_BITS)) | ((uint64_t)r << LSO_STAMP_K_BITS) |
           (uint64_t)(((uint32_t)1 << LSO_STAMP_K_BITS) - 1u - k);
}

typedef struct {
    uint64_t h, s;
} lso_entry;

static int cmp_hash_newest_first(const void* a, const void* b)
{
    const lso_entry* x = (const lso_entry*)a;
    const lso_entry* y = (const lso_entry*)b;
    if (x->h != y->h) return x->h < y->h ? -1 : 1;
    if (x->s != y->s) return x->s > y->s ? -1 : 1;
    return 0;
}

static int cmp_newest_first(const void* a, const void* b)
{
    const lso_entry* x = (const lso_entry*)a;
    const lso_entry* y = (const lso_entry*)b;
    if (x->s != y->s) return x->s > y->s ? -1 : 1;
    return 0;
}

/* in_off/in_hash/in_stamp: the instances' lists (CSR over N).  capacity[i] >= 0.
   chosen[r] outside [0, N) leaves request r out.  out_* receive the new lists,
   each newest first; out_hash/out_stamp must hold sum_i capacity[i] entries.
   Returns 0, or -1 when an argument is out of the stamp layout's range. */
int lso_commit(int32_t N, const int64_t* in_off, const uint64_t* in_hash, const uint64_t* in_stamp,
               const int64_t* capacity, int32_t R, const int64_t* req_off, const uint64_t* req_hashes,
               const int32_t* chosen, uint32_t epoch, int64_t* out_off, uint64_t* out_hash, uint64_t* out_stamp)
{
    if (epoch == 0 || epoch >= ((uint32_t)1 << LSO_STAMP_E_BITS)) return -1;
    if ((int64_t)R > ((int64_t)1 << LSO_STAMP_R_BITS)) return -1;
    for (int32_t r = 0; r < R; ++r)
        if (req_off[r + 1] - req_off[r] > ((int64_t)1 << LSO_STAMP_K_BITS)) return -1;
    out_off[0] = 0;
    for (int32_t i = 0; i < N; ++i) {
        int64_t cnt = in_off[i + 1] - in_off[i];
        for (int32_t r = 0; r < R; ++r)
            if (chosen[r] == i) cnt += req_off[r + 1] - req_off[r];
        lso_entry* A = (lso_entry*)malloc(sizeof(lso_entry) * (size_t)(cnt > 0 ? cnt : 1));
        int64_t m = 0;
        for (int64_t j = in_off[i]; j < in_off[i + 1]; ++j) {
            A[m].h = in_hash[j];
            A[m].s = in_stamp[j];
            ++m;
        }
        for (int32_t r = 0; r < R; ++r) {
            if (chosen[r] != i) continue;
            for (int64_t k = 0; k < req_off[r + 1] - req_off[r]; ++k) {
                A[m].h = req_hashes[req_off[r] + k];
                A[m].s = lso_stamp(epoch, (uint32_t)r, (uint32_t)k);
                ++m;
            }
        }
        /* one entry per block, with its largest stamp */
        qsort(A, (size_t)m, sizeof(lso_entry), cmp_hash_newest_first);
        int64_t u = 0;
        for (int64_t t = 0; t < m; ++t)
            if (u == 0 || A[u - 1].h != A[t].h) A[u++] = A[t];
        /* least recently used out */
        qsort(A, (size_t)u, sizeof(lso_entry), cmp_newest_first);
        int64_t keep = u < capacity[i] ? u : capacity[i];
        for (int64_t t = 0; t < keep; ++t) {
            out_hash[out_off[i] + t] = A[t].h;
            out_stamp[out_off[i] + t] = A[t].s;
        }
        out_off[i + 1] = out_off[i] + keep;
        free(A);
    }
    return 0;
}

int lso_train_round(int mode, int32_t d, int32_t n_hidden, const int32_t* hidden, float* params, const float* mu,
                    const float* inv_sigma, int32_t fifo_cap, int32_t fifo_count, int32_t fifo_head,
                    const float* fifo_x, const float* fifo_y, int32_t rep_count, const float* rep_x,
                    const float* rep_y, int32_t epochs, int32_t batch, float lr, const int32_t* perm,
                    double* loss_out)
{
    return lso_train_round_dropout(mode, d, n_hidden, hidden, params, mu, inv_sigma, fifo_cap, fifo_count, fifo_head,
                                   fifo_x, fifo_y, rep_count, rep_x, rep_y, epochs, batch, lr, perm, 0.0, 0, 0,
                                   loss_out);
}
