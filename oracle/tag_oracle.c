/*
 * Reference oracle for the TAG heterogeneous GNN (graph ingest, forward pass,
 * decision head).  TEST INFRASTRUCTURE ONLY: it exists to check the GPU
 * library.  Only the test suite, the package smoke check and the benchmark's
 * CPU-baseline leg may load it; the product path never does.
 *
 * Plain single-threaded C99, every floating-point quantity in double
 * precision, no blocking, no fusion, no folding of linear maps.  Each
 * function cites the passage of the paper it follows (Section 4.2.1,
 * "Heterogeneous GNN", and Section 4.2, the strategy encoding).
 *
 * Readings of the paper that this file relies on (where the text is silent
 * or garbled) are listed with each function; they are the same readings the
 * GPU library documents.
 *
 * Parity status: every function here is pinned by the CPU test suite against
 * brute force, closed forms, invariants or library routines.  Numeric parity
 * with the paper itself is unpinned: the paper prints no embeddings, scores
 * or worked example.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define TAGO_OK 0
#define TAGO_EINVAL (-1)
#define TAGO_ERANGE (-2)
#define TAGO_EDUP (-3)
#define TAGO_ESHAPE (-4)
#define TAGO_ENOMEM (-7)

typedef struct {
    int32_t f, heads, layers, f_op, f_dev, dec_hidden, bf16;
    double gamma_same, gamma_cross, leaky_slope;
    int32_t sigma;      /* message non-linearity: 0 ReLU, 1 ELU (alpha = 1) */
    int32_t relations;  /* 3: undirected link types (op-op, op-device, device-device);
                           5: directed (op<-op along the tensor, op<-op against it,
                           op<-device, device<-op, device<-device) */
    int32_t edge_act;   /* edge encoders: 0 affine, 1 affine + ReLU */
    int32_t head_mode;  /* 0: K concatenated heads of f/K channels; 1: K heads over all
                           f channels with their own attention vectors, averaged */
} tago_dims;

typedef struct {
    const float *enc_op_w, *enc_op_b, *enc_dev_w, *enc_dev_b;
    const float *enc_edge_w[3], *enc_edge_b[3];
    const float *layer_w, *layer_b, *att_src, *att_dst;
    const float *dec_w1, *dec_b1, *dec_w2, *dec_b2;
} tago_weights;

/* ------------------------------------------------------------------------ */
/* bf16 rounding: round-to-nearest-even of a real number to 8 significand   */
/* bits.  Used only by the bf16 variant of the relation transforms.          */
/* ------------------------------------------------------------------------ */
double tago_round_bf16(double x)
{
    if (x == 0.0 || !isfinite(x)) return x;
    int e;
    double m = frexp(x, &e);            /* x = m * 2^e, 0.5 <= |m| < 1 */
    /* bf16 subnormals (below 2^-126) keep fewer bits: spacing 2^-133 */
    int keep = 8;
    if (e - 1 < -126) keep = 8 - (-126 - (e - 1));
    if (keep < 0) return copysign(0.0, x);
    double r = nearbyint(ldexp(m, keep)); /* default rounding: to nearest, ties even */
    return ldexp(r, e - keep);
}

/* ------------------------------------------------------------------------ */
/* Graph ingest (Section 4.2.1: two node types, three link types).           */
/*                                                                           */
/* The joint graph is turned into four destination buckets:                  */
/*   B0 op  <- op   (tensor links, both directions: neighbour sets are       */
/*                   undirected within a link type)                          */
/*   B1 op  <- dev  (placement links)                                        */
/*   B2 dev <- op   (placement links, other direction)                       */
/*   B3 dev <- dev  (network links, both directions)                         */
/* Each bucket is a CSR keyed by destination; inside a row, entries are      */
/* ordered by (source id, edge id).  Rejected: ids out of range (ERANGE),    */
/* self links and any (destination, source) pair that occurs twice in one    */
/* bucket, which covers duplicate input pairs and a tensor link given in     */
/* both directions (EDUP).  Range errors take precedence.                    */
/* ------------------------------------------------------------------------ */
typedef struct { int32_t row, col, eid; } tago_entry;

static int cmp_entry(const void *pa, const void *pb)
{
    const tago_entry *a = (const tago_entry *)pa, *b = (const tago_entry *)pb;
    if (a->row != b->row) return a->row < b->row ? -1 : 1;
    if (a->col != b->col) return a->col < b->col ? -1 : 1;
    if (a->eid != b->eid) return a->eid < b->eid ? -1 : 1;
    return 0;
}

/* sort the entries, reject repeated (row, col), write the CSR */
static int finish_bucket(tago_entry *ent, int64_t n, int32_t n_rows,
                         int32_t *rowptr, int32_t *col, int32_t *eid)
{
    qsort(ent, (size_t)n, sizeof(tago_entry), cmp_entry);
    int dup = 0;
    for (int64_t i = 1; i < n; ++i)
        if (ent[i].row == ent[i - 1].row && ent[i].col == ent[i - 1].col) dup = 1;
    for (int32_t r = 0; r <= n_rows; ++r) rowptr[r] = 0;
    for (int64_t i = 0; i < n; ++i) rowptr[ent[i].row + 1] += 1;
    for (int32_t r = 0; r < n_rows; ++r) rowptr[r + 1] += rowptr[r];
    for (int64_t i = 0; i < n; ++i) { col[i] = ent[i].col; eid[i] = ent[i].eid; }
    return dup;
}

int tago_csr(int32_t n_op, int32_t n_dev,
             int32_t e_oo, const int32_t *oo_src, const int32_t *oo_dst,
             int32_t e_dd, const int32_t *dd_a, const int32_t *dd_b,
             int32_t e_od, const int32_t *od_op, const int32_t *od_dev,
             int32_t *rp0, int32_t *col0, int32_t *eid0,
             int32_t *rp1, int32_t *col1, int32_t *eid1,
             int32_t *rp2, int32_t *col2, int32_t *eid2,
             int32_t *rp3, int32_t *col3, int32_t *eid3)
{
    if (n_op < 0 || n_dev < 0 || e_oo < 0 || e_dd < 0 || e_od < 0) return TAGO_EINVAL;
    int bad_range = 0, bad_dup = 0;
    for (int32_t i = 0; i < e_oo; ++i) {
        if (oo_src[i] < 0 || oo_src[i] >= n_op || oo_dst[i] < 0 || oo_dst[i] >= n_op) bad_range = 1;
        else if (oo_src[i] == oo_dst[i]) bad_dup = 1;
    }
    for (int32_t i = 0; i < e_dd; ++i) {
        if (dd_a[i] < 0 || dd_a[i] >= n_dev || dd_b[i] < 0 || dd_b[i] >= n_dev) bad_range = 1;
        else if (dd_a[i] == dd_b[i]) bad_dup = 1;
    }
    for (int32_t i = 0; i < e_od; ++i)
        if (od_op[i] < 0 || od_op[i] >= n_op || od_dev[i] < 0 || od_dev[i] >= n_dev) bad_range = 1;
    if (bad_range) return TAGO_ERANGE;

    int64_t cap = 2 * (int64_t)e_oo;
    if (e_od > cap) cap = e_od;
    if (2 * (int64_t)e_dd > cap) cap = 2 * (int64_t)e_dd;
    tago_entry *ent = (tago_entry *)malloc((size_t)(cap > 0 ? cap : 1) * sizeof(tago_entry));
    if (!ent) return TAGO_ENOMEM;

    /* B0: producer p -> consumer c gives (row c, src p) and (row p, src c) */
    for (int32_t i = 0; i < e_oo; ++i) {
        ent[2 * i] = (tago_entry){oo_dst[i], oo_src[i], i};
        ent[2 * i + 1] = (tago_entry){oo_src[i], oo_dst[i], i};
    }
    bad_dup |= finish_bucket(ent, 2 * (int64_t)e_oo, n_op, rp0, col0, eid0);
    /* B1: (op u, device j) gives (row u, src j) */
    for (int32_t i = 0; i < e_od; ++i) ent[i] = (tago_entry){od_op[i], od_dev[i], i};
    bad_dup |= finish_bucket(ent, e_od, n_op, rp1, col1, eid1);
    /* B2: (op u, device j) gives (row j, src u) */
    for (int32_t i = 0; i < e_od; ++i) ent[i] = (tago_entry){od_dev[i], od_op[i], i};
    bad_dup |= finish_bucket(ent, e_od, n_dev, rp2, col2, eid2);
    /* B3: {a, b} gives (row a, src b) and (row b, src a) */
    for (int32_t i = 0; i < e_dd; ++i) {
        ent[2 * i] = (tago_entry){dd_a[i], dd_b[i], i};
        ent[2 * i + 1] = (tago_entry){dd_b[i], dd_a[i], i};
    }
    bad_dup |= finish_bucket(ent, 2 * (int64_t)e_dd, n_dev, rp3, col3, eid3);
    free(ent);
    return bad_dup ? TAGO_EDUP : TAGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Forward pass (Section 4.2.1).                                             */
/*                                                                           */
/* Input encoders: one fully connected layer maps raw node features to      */
/* length f, followed by ReLU; one fully connected layer (no activation)     */
/* maps each raw edge feature to length f.                                   */
/*                                                                           */
/* Layer i, destination u, link type t, neighbour v with edge feature e_uv:  */
/*   z     = W_{i,t} [h_v ; e_uv] + b_{i,t}     (W = [W^h | W^e], f x 2f)   */
/*   m     = sigma(z),   sigma = ReLU                                        */
/*   score = LeakyReLU( a_{i,t}^(k) . m^(k) + adst_{i,t}^(k) . (W^h h_u)^(k) ) */
/*           per attention head k (channels [k f/K, (k+1) f/K))              */
/*   alpha = softmax of the scores over u's neighbours of that link type     */
/*   agg_t = sum alpha * m (per head, heads concatenated)                    */
/*   h'_u  = sum over link types into u of gamma_t * agg_t,                  */
/*           gamma = 1 between same-type nodes, 0.1 between op and device.   */
/* No self loop, residual or normalisation.  An empty bucket adds zero.      */
/* bf16 variant: h and W^h are rounded to bf16 before the W^h product and    */
/* the product W^h h is rounded to bf16 after it; all else stays double.     */
/*                                                                           */
/* Readings where the paper leaves a choice (defaults first):                */
/*  - link types: three undirected relations (op-op, op-device, device-      */
/*    device; both ends of a link share W), or five directed ones (op<-op    */
/*    along the tensor, op<-op against it, op<-device, device<-op,           */
/*    device<-device), each with its own W, b, a, adst;                      */
/*  - edge encoders: affine, or affine followed by ReLU;                     */
/*  - heads: K concatenated heads of f/K channels, or K heads over all f     */
/*    channels (attention vectors a, adst of length f per head) averaged.    */
/* ------------------------------------------------------------------------ */
static double leaky(double x, double slope) { return x > 0.0 ? x : slope * x; }

/* one destination row of one bucket: adds gamma * agg into out[f].
 * Concatenated heads (head_mode 0): head k scores and aggregates channels
 * [k f/K, (k+1) f/K) with a_src, a_dst of length f.  Averaged full-width
 * heads (head_mode 1): head k scores all f channels with its own vectors
 * a_src + k f, a_dst + k f, and the K aggregates are averaged. */
static void aggregate_row(const tago_dims *d, int32_t beg, int32_t end,
                          const int32_t *col, const int32_t *eid,
                          const double *ysrc,       /* [n_src][f]  W^h h_v  */
                          const double *ydst_u,     /* [f]         W^h h_u  */
                          const double *edge_term,  /* per eid [f]: W^e e + b */
                          const uint8_t *od_bits,   /* od: eid -> bit selects edge_term row */
                          const float *a_src, const float *a_dst,
                          double gamma, double *out, double *scratch_m, double *scratch_s,
                          double *alpha_out)
{
    const int f = d->f, K = d->heads, avg = d->head_mode == 1, dh = avg ? f : f / K;
    const double g = avg ? gamma / K : gamma;
    const int32_t n = end - beg;
    if (n == 0) return;
    for (int32_t e = 0; e < n; ++e) {
        const int32_t v = col[beg + e];
        const int32_t id = eid[beg + e];
        const double *te = od_bits ? edge_term + (size_t)od_bits[id] * f : edge_term + (size_t)id * f;
        for (int c = 0; c < f; ++c) {
            double z = ysrc[(size_t)v * f + c] + te[c];
            /* sigma of the layer equation (Section 4.2.1): ReLU, or ELU as a variant */
            scratch_m[(size_t)e * f + c] = z > 0.0 ? z : (d->sigma == 1 ? expm1(z) : 0.0);
        }
    }
    for (int k = 0; k < K; ++k) {
        const int c0 = avg ? 0 : k * dh, c1 = c0 + dh;
        const float *as = avg ? a_src + (size_t)k * f : a_src;
        const float *ad = avg ? a_dst + (size_t)k * f : a_dst;
        double qd = 0.0;
        for (int c = c0; c < c1; ++c) qd += (double)ad[c] * ydst_u[c];
        double mx = -INFINITY;
        for (int32_t e = 0; e < n; ++e) {
            double s = 0.0;
            for (int c = c0; c < c1; ++c) s += (double)as[c] * scratch_m[(size_t)e * f + c];
            s = leaky(s + qd, d->leaky_slope);
            scratch_s[e] = s;
            if (s > mx) mx = s;
        }
        double z = 0.0;
        for (int32_t e = 0; e < n; ++e) z += exp(scratch_s[e] - mx);
        for (int32_t e = 0; e < n; ++e) {
            double al = exp(scratch_s[e] - mx) / z;
            if (alpha_out) alpha_out[(size_t)(beg + e) * K + k] = al;
            for (int c = c0; c < c1; ++c)
                out[c] += g * al * scratch_m[(size_t)e * f + c];
        }
    }
}

/* y[n][f] = W^h x[n][f], W^h = columns [0, f) of the f x 2f row-major W.
 * bf16 variant: both operands are rounded to bf16 first, the sum is rounded
 * after (the operands are rounded once, before the loops, into copies). */
static void apply_wh(int f, int32_t n, const float *W, const double *x, double *y, int bf16)
{
    double *wr = malloc(sizeof(double) * (size_t)f * f);
    double *hr = malloc(sizeof(double) * (size_t)f);
    if (!wr || !hr) { free(wr); free(hr); return; }
    for (int c = 0; c < f; ++c)
        for (int k = 0; k < f; ++k) {
            double w = W[(size_t)c * 2 * f + k];
            wr[(size_t)c * f + k] = bf16 ? tago_round_bf16(w) : w;
        }
    for (int32_t v = 0; v < n; ++v) {
        for (int k = 0; k < f; ++k) {
            double h = x[(size_t)v * f + k];
            hr[k] = bf16 ? tago_round_bf16(h) : h;
        }
        for (int c = 0; c < f; ++c) {
            double s = 0.0;
            for (int k = 0; k < f; ++k) s += wr[(size_t)c * f + k] * hr[k];
            y[(size_t)v * f + c] = bf16 ? tago_round_bf16(s) : s;
        }
    }
    free(wr); free(hr);
}

/* te[n][f] = W^e enc[n][f] + b, W^e = columns [f, 2f) */
static void apply_we(int f, int32_t n, const float *W, const float *b, const double *enc, double *te)
{
    for (int32_t i = 0; i < n; ++i)
        for (int c = 0; c < f; ++c) {
            double s = b[c];
            for (int k = 0; k < f; ++k) s += (double)W[(size_t)c * 2 * f + f + k] * enc[(size_t)i * f + k];
            te[(size_t)i * f + c] = s;
        }
}

/* one fully connected layer on raw features: out[n][f] = A x + c (ReLU optional) */
static void encode(int f, int32_t n, int din, const float *A, const float *c,
                   const float *x, double *out, int relu)
{
    for (int32_t i = 0; i < n; ++i)
        for (int o = 0; o < f; ++o) {
            double s = c[o];
            for (int t = 0; t < din; ++t) s += (double)A[(size_t)o * din + t] * (double)x[(size_t)i * din + t];
            out[(size_t)i * f + o] = (relu && s < 0.0) ? 0.0 : s;
        }
}

/* B0 split by direction for the directed reading: forward entries (row =
 * consumer, src = producer) and backward entries (row = producer, src =
 * consumer), each sorted by (source, edge id).  Links were validated by
 * tago_csr. */
static int directed_op_buckets(int32_t n_op, int32_t e_oo, const int32_t *oo_src, const int32_t *oo_dst,
                               int32_t *rpf, int32_t *colf, int32_t *eidf,
                               int32_t *rpb, int32_t *colb, int32_t *eidb)
{
    tago_entry *ent = (tago_entry *)malloc((size_t)(e_oo > 0 ? e_oo : 1) * sizeof(tago_entry));
    if (!ent) return TAGO_ENOMEM;
    for (int32_t i = 0; i < e_oo; ++i) ent[i] = (tago_entry){oo_dst[i], oo_src[i], i};
    finish_bucket(ent, e_oo, n_op, rpf, colf, eidf);
    for (int32_t i = 0; i < e_oo; ++i) ent[i] = (tago_entry){oo_src[i], oo_dst[i], i};
    finish_bucket(ent, e_oo, n_op, rpb, colb, eidb);
    free(ent);
    return TAGO_OK;
}

int tago_forward(const tago_dims *d,
                 int32_t n_op, int32_t n_dev,
                 int32_t e_oo, const int32_t *oo_src, const int32_t *oo_dst,
                 int32_t e_dd, const int32_t *dd_a, const int32_t *dd_b,
                 int32_t e_od, const int32_t *od_op, const int32_t *od_dev,
                 const float *x_op, const float *x_dev, const float *x_oo,
                 const float *x_dd, const uint8_t *x_od,
                 const tago_weights *w,
                 double *E_op, double *E_dev,
                 double *alpha_layer0 /* optional: [T][K], buckets B0,B1,B2,B3 concatenated
                                         (three undirected relations only) */)
{
    if (!d || !w || d->f <= 0 || d->heads <= 0 || d->layers < 0) return TAGO_ESHAPE;
    if (d->relations != 3 && d->relations != 5) return TAGO_ESHAPE;
    if (d->head_mode != 0 && d->head_mode != 1) return TAGO_ESHAPE;
    if (d->edge_act != 0 && d->edge_act != 1) return TAGO_ESHAPE;
    if (d->head_mode == 0 && d->f % d->heads) return TAGO_ESHAPE;
    const int f = d->f, NR = d->relations;
    const size_t asz = (size_t)(d->head_mode == 1 ? d->heads : 1) * f;   /* attention vector length */
    if (NR == 5) alpha_layer0 = NULL;
    int st = TAGO_OK;
    const int64_t nn0 = 2 * (int64_t)e_oo, nn1 = e_od, nn3 = 2 * (int64_t)e_dd;
    int32_t *rp0 = malloc(sizeof(int32_t) * (n_op + 1)), *rp1 = malloc(sizeof(int32_t) * (n_op + 1));
    int32_t *rp2 = malloc(sizeof(int32_t) * (n_dev + 1)), *rp3 = malloc(sizeof(int32_t) * (n_dev + 1));
    int32_t *c0 = malloc(sizeof(int32_t) * (nn0 + 1)), *i0 = malloc(sizeof(int32_t) * (nn0 + 1));
    int32_t *c1 = malloc(sizeof(int32_t) * (nn1 + 1)), *i1 = malloc(sizeof(int32_t) * (nn1 + 1));
    int32_t *c2 = malloc(sizeof(int32_t) * (nn1 + 1)), *i2 = malloc(sizeof(int32_t) * (nn1 + 1));
    int32_t *c3 = malloc(sizeof(int32_t) * (nn3 + 1)), *i3 = malloc(sizeof(int32_t) * (nn3 + 1));
    /* directed reading: op<-op split into forward (along the tensor) and backward */
    int32_t *rpf = malloc(sizeof(int32_t) * (n_op + 1)), *rpb = malloc(sizeof(int32_t) * (n_op + 1));
    int32_t *cf = malloc(sizeof(int32_t) * ((size_t)e_oo + 1)), *idf = malloc(sizeof(int32_t) * ((size_t)e_oo + 1));
    int32_t *cb = malloc(sizeof(int32_t) * ((size_t)e_oo + 1)), *idb = malloc(sizeof(int32_t) * ((size_t)e_oo + 1));
    double *h_op = calloc((size_t)n_op * f + 1, sizeof(double));
    double *h_dev = calloc((size_t)n_dev * f + 1, sizeof(double));
    double *nh_op = calloc((size_t)n_op * f + 1, sizeof(double));
    double *nh_dev = calloc((size_t)n_dev * f + 1, sizeof(double));
    double *ys_op = calloc((size_t)n_op * f + 1, sizeof(double));    /* W^h h of a relation's sources */
    double *ys_dev = calloc((size_t)n_dev * f + 1, sizeof(double));
    double *yd_op = calloc((size_t)n_op * f + 1, sizeof(double));    /* W^h h of its destinations */
    double *yd_dev = calloc((size_t)n_dev * f + 1, sizeof(double));
    double *enc_oo = calloc((size_t)e_oo * f + 1, sizeof(double));
    double *enc_dd = calloc((size_t)e_dd * f + 1, sizeof(double));
    double *enc_od = calloc((size_t)2 * f, sizeof(double));
    double *te_oo = calloc((size_t)e_oo * f + 1, sizeof(double));
    double *te_dd = calloc((size_t)e_dd * f + 1, sizeof(double));
    double *te_od = calloc((size_t)2 * f, sizeof(double));
    int64_t maxdeg = 1;
    double *sm = NULL, *ss = NULL;
    float *xbit = malloc(sizeof(float) * 2);
    uint8_t *bit_of = malloc((size_t)nn1 + 1);
    if (!rp0 || !rp1 || !rp2 || !rp3 || !c0 || !i0 || !c1 || !i1 || !c2 || !i2 || !c3 || !i3 || !rpf ||
        !rpb || !cf || !idf || !cb || !idb || !h_op || !h_dev || !nh_op || !nh_dev || !ys_op || !ys_dev ||
        !yd_op || !yd_dev || !enc_oo || !enc_dd || !enc_od || !te_oo || !te_dd || !te_od || !xbit || !bit_of) {
        st = TAGO_ENOMEM; goto done;
    }

    st = tago_csr(n_op, n_dev, e_oo, oo_src, oo_dst, e_dd, dd_a, dd_b, e_od, od_op, od_dev,
                  rp0, c0, i0, rp1, c1, i1, rp2, c2, i2, rp3, c3, i3);
    if (st != TAGO_OK) goto done;
    if (NR == 5) {
        st = directed_op_buckets(n_op, e_oo, oo_src, oo_dst, rpf, cf, idf, rpb, cb, idb);
        if (st != TAGO_OK) goto done;
    }
    for (int32_t r = 0; r < n_op; ++r) {
        if (rp0[r + 1] - rp0[r] > maxdeg) maxdeg = rp0[r + 1] - rp0[r];
        if (rp1[r + 1] - rp1[r] > maxdeg) maxdeg = rp1[r + 1] - rp1[r];
    }
    for (int32_t r = 0; r < n_dev; ++r) {
        if (rp2[r + 1] - rp2[r] > maxdeg) maxdeg = rp2[r + 1] - rp2[r];
        if (rp3[r + 1] - rp3[r] > maxdeg) maxdeg = rp3[r + 1] - rp3[r];
    }
    sm = malloc(sizeof(double) * (size_t)maxdeg * f);
    ss = malloc(sizeof(double) * (size_t)maxdeg);
    if (!sm || !ss) { st = TAGO_ENOMEM; goto done; }
    for (int64_t i = 0; i < nn1; ++i) bit_of[i] = x_od[i] ? 1 : 0;

    /* input encoders (edge encoders: affine, or affine + ReLU) */
    encode(f, n_op, d->f_op, w->enc_op_w, w->enc_op_b, x_op, h_op, 1);
    encode(f, n_dev, d->f_dev, w->enc_dev_w, w->enc_dev_b, x_dev, h_dev, 1);
    encode(f, e_oo, 1, w->enc_edge_w[0], w->enc_edge_b[0], x_oo, enc_oo, d->edge_act);
    encode(f, e_dd, 2, w->enc_edge_w[2], w->enc_edge_b[2], x_dd, enc_dd, d->edge_act);
    /* the op-device edge feature is a single placement bit: encode both values */
    xbit[0] = 0.0f; xbit[1] = 1.0f;
    encode(f, 2, 1, w->enc_edge_w[1], w->enc_edge_b[1], xbit, enc_od, d->edge_act);

    for (int layer = 0; layer < d->layers; ++layer) {
        const float *W[5], *bb[5], *as[5], *ad[5];
        for (int r = 0; r < NR; ++r) {
            W[r] = w->layer_w + ((size_t)layer * NR + r) * f * 2 * f;
            bb[r] = w->layer_b + ((size_t)layer * NR + r) * f;
            as[r] = w->att_src + ((size_t)layer * NR + r) * asz;
            ad[r] = w->att_dst + ((size_t)layer * NR + r) * asz;
        }
        double *alpha = (layer == 0) ? alpha_layer0 : NULL;
        const int64_t off1 = nn0, off2 = nn0 + nn1, off3 = nn0 + 2 * nn1;
        memset(nh_op, 0, sizeof(double) * (size_t)n_op * f);
        memset(nh_dev, 0, sizeof(double) * (size_t)n_dev * f);

        if (NR == 3) {
            /* op <- op (tensor links, both directions, one relation) */
            apply_we(f, e_oo, W[0], bb[0], enc_oo, te_oo);
            apply_wh(f, n_op, W[0], h_op, ys_op, d->bf16);
            for (int32_t u = 0; u < n_op; ++u)
                aggregate_row(d, rp0[u], rp0[u + 1], c0, i0, ys_op, ys_op + (size_t)u * f, te_oo, NULL,
                              as[0], ad[0], d->gamma_same, nh_op + (size_t)u * f, sm, ss, alpha);
            /* placement links: W^h_od applies to both node types */
            apply_we(f, 2, W[1], bb[1], enc_od, te_od);
            apply_wh(f, n_op, W[1], h_op, ys_op, d->bf16);
            apply_wh(f, n_dev, W[1], h_dev, ys_dev, d->bf16);
            for (int32_t u = 0; u < n_op; ++u)   /* op <- device */
                aggregate_row(d, rp1[u], rp1[u + 1], c1, i1, ys_dev, ys_op + (size_t)u * f, te_od, bit_of,
                              as[1], ad[1], d->gamma_cross, nh_op + (size_t)u * f, sm, ss,
                              alpha ? alpha + (size_t)off1 * d->heads : NULL);
            for (int32_t j = 0; j < n_dev; ++j)  /* device <- op */
                aggregate_row(d, rp2[j], rp2[j + 1], c2, i2, ys_op, ys_dev + (size_t)j * f, te_od, bit_of,
                              as[1], ad[1], d->gamma_cross, nh_dev + (size_t)j * f, sm, ss,
                              alpha ? alpha + (size_t)off2 * d->heads : NULL);
            /* device <- device (network links) */
            apply_we(f, e_dd, W[2], bb[2], enc_dd, te_dd);
            apply_wh(f, n_dev, W[2], h_dev, ys_dev, d->bf16);
            for (int32_t j = 0; j < n_dev; ++j)
                aggregate_row(d, rp3[j], rp3[j + 1], c3, i3, ys_dev, ys_dev + (size_t)j * f, te_dd, NULL,
                              as[2], ad[2], d->gamma_same, nh_dev + (size_t)j * f, sm, ss,
                              alpha ? alpha + (size_t)off3 * d->heads : NULL);
        } else {
            /* relation 0: op <- op along the tensor (row = consumer) */
            apply_we(f, e_oo, W[0], bb[0], enc_oo, te_oo);
            apply_wh(f, n_op, W[0], h_op, ys_op, d->bf16);
            for (int32_t u = 0; u < n_op; ++u)
                aggregate_row(d, rpf[u], rpf[u + 1], cf, idf, ys_op, ys_op + (size_t)u * f, te_oo, NULL,
                              as[0], ad[0], d->gamma_same, nh_op + (size_t)u * f, sm, ss, NULL);
            /* relation 1: op <- op against the tensor (row = producer) */
            apply_we(f, e_oo, W[1], bb[1], enc_oo, te_oo);
            apply_wh(f, n_op, W[1], h_op, ys_op, d->bf16);
            for (int32_t u = 0; u < n_op; ++u)
                aggregate_row(d, rpb[u], rpb[u + 1], cb, idb, ys_op, ys_op + (size_t)u * f, te_oo, NULL,
                              as[1], ad[1], d->gamma_same, nh_op + (size_t)u * f, sm, ss, NULL);
            /* relation 2: op <- device (W_2 on device sources and op destinations) */
            apply_we(f, 2, W[2], bb[2], enc_od, te_od);
            apply_wh(f, n_dev, W[2], h_dev, ys_dev, d->bf16);
            apply_wh(f, n_op, W[2], h_op, yd_op, d->bf16);
            for (int32_t u = 0; u < n_op; ++u)
                aggregate_row(d, rp1[u], rp1[u + 1], c1, i1, ys_dev, yd_op + (size_t)u * f, te_od, bit_of,
                              as[2], ad[2], d->gamma_cross, nh_op + (size_t)u * f, sm, ss, NULL);
            /* relation 3: device <- op (W_3 on op sources and device destinations) */
            apply_we(f, 2, W[3], bb[3], enc_od, te_od);
            apply_wh(f, n_op, W[3], h_op, ys_op, d->bf16);
            apply_wh(f, n_dev, W[3], h_dev, yd_dev, d->bf16);
            for (int32_t j = 0; j < n_dev; ++j)
                aggregate_row(d, rp2[j], rp2[j + 1], c2, i2, ys_op, yd_dev + (size_t)j * f, te_od, bit_of,
                              as[3], ad[3], d->gamma_cross, nh_dev + (size_t)j * f, sm, ss, NULL);
            /* relation 4: device <- device */
            apply_we(f, e_dd, W[4], bb[4], enc_dd, te_dd);
            apply_wh(f, n_dev, W[4], h_dev, ys_dev, d->bf16);
            for (int32_t j = 0; j < n_dev; ++j)
                aggregate_row(d, rp3[j], rp3[j + 1], c3, i3, ys_dev, ys_dev + (size_t)j * f, te_dd, NULL,
                              as[4], ad[4], d->gamma_same, nh_dev + (size_t)j * f, sm, ss, NULL);
        }
        memcpy(h_op, nh_op, sizeof(double) * (size_t)n_op * f);
        memcpy(h_dev, nh_dev, sizeof(double) * (size_t)n_dev * f);
    }
    memcpy(E_op, h_op, sizeof(double) * (size_t)n_op * f);
    memcpy(E_dev, h_dev, sizeof(double) * (size_t)n_dev * f);

done:
    free(rp0); free(rp1); free(rp2); free(rp3); free(c0); free(i0); free(c1); free(i1);
    free(c2); free(i2); free(c3); free(i3); free(rpf); free(rpb); free(cf); free(idf); free(cb); free(idb);
    free(h_op); free(h_dev); free(nh_op); free(nh_dev);
    free(ys_op); free(ys_dev); free(yd_op); free(yd_dev); free(enc_oo); free(enc_dd); free(enc_od); free(te_oo);
    free(te_dd); free(te_od); free(sm); free(ss); free(xbit); free(bit_of);
    return st;
}

/* ------------------------------------------------------------------------ */
/* Decision head (Section 4.2.1, the decoder after the GNN; Section 4.2,     */
/* the strategy encoding P and O).                                           */
/*                                                                           */
/* For op i and strategy slice a = (placement row P_i = mask, option O_i):   */
/*   x = [ sum_j P_ij E_dev[j] ; E_op[i] ; onehot(O_i) ]   (length 2f + 4)   */
/*   score = w2 . ReLU(W1 x + b1) + b2   (hidden width H > 0), or            */
/*   score = w2 . x + b2                 (H = 0, the literal linear Dense)   */
/*   prior = softmax of the scores over the slice table, argmax = first max. */
/* Mask bits at or above the device count are ignored.                       */
/* Decoded decision: option 0 replicate + AllReduce, 1 replicate + PS,       */
/* 2 duplicate (sufficient-factor broadcasting, no gradient sync), 3 model   */
/* parallel.  replicas = popcount(mask) for options 0-2, 1 for option 3;     */
/* sync = 0 AllReduce, 1 PS, 2 none; sfb = (option == 2).                    */
/* ------------------------------------------------------------------------ */
int tago_decide(const tago_dims *d, int32_t n_op, int32_t n_dev,
                const double *E_op, const double *E_dev,
                int32_t n_slices, const uint64_t *mask, const uint8_t *option,
                int32_t n_query, const int32_t *query_op,
                const tago_weights *w,
                int32_t *argmax, double *best, double *prior /* [Q][S] or NULL */,
                uint64_t *dec_mask, int32_t *dec_replicas, int32_t *dec_option,
                int32_t *dec_sync, int32_t *dec_sfb)
{
    const int f = d->f, H = d->dec_hidden, din = 2 * f + 4;
    if (n_slices <= 0 || n_query < 0) return TAGO_EINVAL;
    for (int32_t a = 0; a < n_slices; ++a) if (option[a] > 3) return TAGO_ERANGE;
    for (int32_t q = 0; q < n_query; ++q) if (query_op[q] < 0 || query_op[q] >= n_op) return TAGO_ERANGE;
    double *x = malloc(sizeof(double) * din);
    double *sc = malloc(sizeof(double) * n_slices);
    if (!x || !sc) { free(x); free(sc); return TAGO_ENOMEM; }
    for (int32_t q = 0; q < n_query; ++q) {
        const int32_t i = query_op[q];
        for (int32_t a = 0; a < n_slices; ++a) {
            for (int t = 0; t < din; ++t) x[t] = 0.0;
            for (int32_t j = 0; j < n_dev && j < 64; ++j)
                if ((mask[a] >> j) & 1u)
                    for (int c = 0; c < f; ++c) x[c] += E_dev[(size_t)j * f + c];
            for (int c = 0; c < f; ++c) x[f + c] = E_op[(size_t)i * f + c];
            x[2 * f + option[a]] = 1.0;
            double s = w->dec_b2[0];
            if (H > 0) {
                for (int h = 0; h < H; ++h) {
                    double t = w->dec_b1[h];
                    for (int k = 0; k < din; ++k) t += (double)w->dec_w1[(size_t)h * din + k] * x[k];
                    if (t > 0.0) s += (double)w->dec_w2[h] * t;
                }
            } else {
                for (int k = 0; k < din; ++k) s += (double)w->dec_w2[k] * x[k];
            }
            sc[a] = s;
        }
        int32_t am = 0;
        for (int32_t a = 1; a < n_slices; ++a) if (sc[a] > sc[am]) am = a;
        argmax[q] = am;
        best[q] = sc[am];
        if (prior) {
            double z = 0.0;
            for (int32_t a = 0; a < n_slices; ++a) z += exp(sc[a] - sc[am]);
            for (int32_t a = 0; a < n_slices; ++a) prior[(size_t)q * n_slices + a] = exp(sc[a] - sc[am]) / z;
        }
        {
            uint64_t valid = n_dev >= 64 ? ~(uint64_t)0 : (((uint64_t)1 << n_dev) - 1);
            uint64_t m = mask[am] & valid;
            int pc = 0;
            for (int j = 0; j < 64; ++j) pc += (int)((m >> j) & 1u);
            int o = option[am];
            if (dec_mask) dec_mask[q] = m;
            if (dec_option) dec_option[q] = o;
            if (dec_replicas) dec_replicas[q] = (o == 3) ? 1 : pc;
            if (dec_sync) dec_sync[q] = (o == 0) ? 0 : (o == 1) ? 1 : 2;
            if (dec_sfb) dec_sfb[q] = (o == 2);
        }
    }
    free(x); free(sc);
    return TAGO_OK;
}
