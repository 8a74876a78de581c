/*
 * tag.h -- C ABI of the MI355X (gfx950) heterogeneous-GNN hot path of TAG's
 * strategy search ("Expediting Distributed DNN Training with Device
 * Topology-Aware Graph Deployment", arXiv 2302.06126).
 *
 * Three stages, each backed by hand-written HIP kernels:
 *   tag_graph_build  relation-bucketed CSR of the joint op/device graph
 *                    (Section 4.2.1: two node types, three link types)
 *   tag_gnn_forward  encoders + L heterogeneous GAT layers over a batch of
 *                    candidate strategies (Section 4.2.1, layer equation and
 *                    multi-head attention aggregation with gamma weights)
 *   tag_gnn_decide   per-op decision head over strategy slices (Section
 *                    4.2.1, decoder; Section 4.2, placement P and the four
 *                    replication options O)
 *
 * Conventions shared by every call:
 *  - The library never allocates device memory.  All buffers are caller
 *    owned; `tag_graph_plan`, `tag_gnn_workspace` and
 *    `tag_gnn_decide_workspace` give their sizes.  (The one exception is
 *    the static scratch array of `tag_gnn_decide_noalloc`, part of the
 *    library's code object.)  Pointers documented as
 *    DEVICE must be device (or managed) memory, 256-byte alignment is
 *    recommended and 16-byte alignment is required.
 *  - `hip_stream` is a hipStream_t passed as void* (NULL = legacy stream).
 *  - Every function returns a tag_status.  Arguments are validated on the
 *    host before anything is enqueued; on a non-OK status nothing has been
 *    enqueued and `tag_last_error()` (thread-local) describes the problem.
 *  - tag_gnn_forward and tag_gnn_decide are asynchronous on `hip_stream`.
 *    tag_graph_build synchronises the stream once, to read the device-side
 *    validation result.
 *  - No exceptions cross this ABI.
 */
#ifndef TAG_H
#define TAG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tag_status;
#define TAG_OK 0
#define TAG_EINVAL (-1)   /* null pointer, negative size, bad enum value      */
#define TAG_ERANGE (-2)   /* node id out of range for its topology            */
#define TAG_EDUP (-3)     /* self link, or a (destination, source) pair twice  */
                          /* in one bucket: duplicate pair, or a tensor link   */
                          /* given in both directions                          */
#define TAG_ESHAPE (-4)   /* unsupported dimensions (see tag_model_dims)      */
#define TAG_ENOSPACE (-5) /* caller buffer or workspace too small             */
#define TAG_EHIP (-6)     /* HIP runtime or launch error                      */

typedef enum { TAG_F32 = 0, TAG_BF16 = 1 } tag_dtype;

/* Relations (link types), in the order every per-relation array uses. */
enum { TAG_REL_OO = 0, TAG_REL_OD = 1, TAG_REL_DD = 2 };
/* Destination buckets produced by tag_graph_build. */
enum { TAG_B_OP_OP = 0, TAG_B_OP_DEV = 1, TAG_B_DEV_OP = 2, TAG_B_DEV_DEV = 3 };

/* ------------------------------------------------------------------------ */
/* Graph ingest                                                              */
/* ------------------------------------------------------------------------ */

/*
 * A batch of G >= 1 disjoint topologies (joint op/device graphs).  Node ids in
 * the edge arrays are LOCAL to their topology; topology g's op->op links are
 * entries [oo_off[g], oo_off[g+1]) of oo_src/oo_dst, and likewise for the
 * other two link types.  In the built graph, topology g's ops are global rows
 * [sum_{h<g} n_op[h], ...) and its devices likewise.
 *
 *   op->op      (oo_src[i] -> oo_dst[i]): a tensor from producer to consumer.
 *               Neighbour sets are undirected, so the link feeds both ends.
 *   dev-dev     {dd_a[i], dd_b[i]}: an unordered network link (either order).
 *   op-dev      (od_op[i], od_dev[i]): a possible placement of the op group on
 *               the device group; it carries the placement bit at run time.
 *               Any subset of the N x M pairs may be given.
 *
 * Rejected by tag_graph_build: ids outside [0, n) of their topology
 * (TAG_ERANGE, takes precedence), self links, and any pair given twice
 * (including p->c together with c->p) (TAG_EDUP).
 */
typedef struct tag_graph_desc {
    int32_t n_graphs;           /* G >= 1                                       */
    const int32_t *n_op;        /* HOST [G]  ops per topology, >= 1             */
    const int32_t *n_dev;       /* HOST [G]  devices per topology, 1..64        */
    const int64_t *oo_off;      /* HOST [G+1] prefix offsets, oo_off[0] = 0     */
    const int64_t *dd_off;      /* HOST [G+1]                                   */
    const int64_t *od_off;      /* HOST [G+1]                                   */
    const int32_t *oo_src, *oo_dst;  /* DEVICE [E_oo]                           */
    const int32_t *dd_a, *dd_b;      /* DEVICE [E_dd]                           */
    const int32_t *od_op, *od_dev;   /* DEVICE [E_od]                           */
} tag_graph_desc;

typedef struct tag_graph tag_graph;   /* opaque host handle */

/* Sizes of the caller buffers tag_graph_build needs (bytes).  Host only. */
tag_status tag_graph_plan(const tag_graph_desc *desc, size_t *csr_bytes, size_t *tmp_bytes);

/*
 * Builds the four destination buckets (CSR keyed by destination, entries of
 * a row ordered by (source id, edge id); ids global):
 *   B0 op<-op  (2 E_oo entries)   B1 op<-dev (E_od)
 *   B2 dev<-op (E_od)             B3 dev<-dev (2 E_dd)
 * csr_buf (DEVICE, csr_bytes) holds the result and must outlive the handle;
 * tmp_buf (DEVICE, tmp_bytes) is scratch, free after return.  The edge
 * arrays are read only during the call.  On success *out receives a handle;
 * on failure *out is NULL.  Synchronises hip_stream once.
 */
tag_status tag_graph_build(const tag_graph_desc *desc, void *csr_buf, size_t csr_bytes,
                           void *tmp_buf, size_t tmp_bytes, void *hip_stream, tag_graph **out);

/* Sizes of the built graph: nodes and entries per bucket.  Host only. */
typedef struct tag_graph_info {
    int32_t n_graphs, max_dev;          /* max_dev = largest per-topology device count */
    int64_t n_op, n_dev;                /* totals over the G topologies                */
    int64_t e_oo, e_dd, e_od;           /* input link counts                           */
    int64_t rows[4], nnz[4];            /* per bucket                                  */
    int32_t max_degree[4];              /* per bucket                                  */
} tag_graph_info;
tag_status tag_graph_get_info(const tag_graph *g, tag_graph_info *info);

/* Copies one bucket to HOST arrays rowptr[rows+1], col[nnz], eid[nnz]
 * (any may be NULL).  Synchronous; for checking and debugging. */
tag_status tag_graph_export(const tag_graph *g, int32_t bucket, int32_t *rowptr_host,
                            int32_t *col_host, int32_t *eid_host);

/* Frees the host handle.  The caller's buffers are untouched. */
void tag_graph_destroy(tag_graph *g);

/* ------------------------------------------------------------------------ */
/* Forward pass                                                              */
/* ------------------------------------------------------------------------ */

/*
 * Model dimensions.
 *   f           hidden width, one of 64, 128, 256
 *   heads       attention heads K: power of two, 1..64; head k owns channels
 *               [k f/K, (k+1) f/K) and heads are concatenated
 *   layers      L, 1..16
 *   f_op        raw op feature width, 1..64
 *   f_dev       raw device feature width, 1..64
 *   dec_hidden  decoder hidden width H: 0 = a single linear Dense layer,
 *               else 1..1024 (Dense + ReLU + scalar readout)
 *   dtype       TAG_F32: everything fp32.  TAG_BF16: the relation transforms
 *               W^h h take bf16 operands (round-to-nearest-even) with fp32
 *               accumulation and store W^h h and the hidden embeddings in
 *               bf16; attention and aggregation stay fp32.
 *   gamma_same  gamma for op-op and device-device links (paper: 1)
 *   gamma_cross gamma for op-device links (paper: 0.1)
 *   leaky_slope LeakyReLU slope of the attention score, in [0, 1] (GAT: 0.2)
 *   sigma       the message non-linearity sigma of the layer equation, which
 *               the paper leaves open: 0 ReLU, 1 ELU (x > 0 ? x : e^x - 1)
 */
typedef struct tag_model_dims {
    int32_t f, heads, layers, f_op, f_dev, dec_hidden;
    int32_t dtype;
    float gamma_same, gamma_cross, leaky_slope;
    int32_t sigma;   /* message non-linearity: 0 ReLU (default), 1 ELU with   */
                     /* alpha = 1 (a variant; needs dtype TAG_F32)           */
    /* Readings of Section 4.2.1 that the paper leaves open.  0 = default.  */
    /* The three variants run on a generic fp32 path (dtype TAG_F32, ReLU   */
    /* messages, no training step).                                         */
    int32_t relations;  /* 0 or 3: three undirected link types (R = 3).     */
                        /* 5: directed relations (R = 5) in this order:     */
                        /* op<-op along the tensor (row = consumer), op<-op */
                        /* against it (row = producer), op<-device,         */
                        /* device<-op, device<-device; each has its own W,  */
                        /* b, a, adst and softmax; gamma as for its types.  */
    int32_t edge_act;   /* 0: affine edge encoders e = A x + c;             */
                        /* 1: e = ReLU(A x + c)                             */
    int32_t head_mode;  /* 0: K concatenated heads of f/K channels;         */
                        /* 1: K heads over all f channels, each with its    */
                        /* own attention vectors, averaged (K <= 8)         */
} tag_model_dims;

/*
 * Parameters, all DEVICE fp32, row-major, caller owned.
 *   enc_op_w [f][f_op], enc_op_b [f]        op encoder, h0 = ReLU(A x + c)
 *   enc_dev_w [f][f_dev], enc_dev_b [f]     device encoder
 *   enc_edge_w[r] [f][d_r], enc_edge_b[r] [f]  edge encoder of relation r,
 *                                           e = A x + c (no activation);
 *                                           d = 1 (oo), 1 (od), 2 (dd)
 *   layer_w [L][R][f][2f]                   W_{l,r} = [W^h | W^e] acting on
 *                                           the concatenation [h_v ; e_uv]
 *                                           (R = 3, or 5 with relations = 5)
 *   layer_b [L][R][f]                       b_{l,r}
 *   att_src [L][R][f]                       message attention vector a_{l,r}
 *                                           ([L][R][K][f] with head_mode = 1)
 *   att_dst [L][R][f]                       destination attention vector,
 *                                           applied to W^h_{l,r} h_u (same
 *                                           shape as att_src)
 *   dec_w1 [H][2f+4], dec_b1 [H], dec_w2 [H], dec_b2 [1]   decoder (H > 0)
 *   dec_w2 [2f+4], dec_b2 [1]               decoder (H = 0; w1, b1 unused)
 * Decoder input order: [sum_j P_ij E_dev[j] ; E_op[i] ; onehot(option)].
 */
typedef struct tag_weights {
    const float *enc_op_w, *enc_op_b, *enc_dev_w, *enc_dev_b;
    const float *enc_edge_w[3], *enc_edge_b[3];
    const float *layer_w, *layer_b, *att_src, *att_dst;
    const float *dec_w1, *dec_b1, *dec_w2, *dec_b2;
} tag_weights;

/*
 * Per-candidate inputs for R replicas of the built graph (R candidate
 * strategies sharing each topology; candidate (r, g) is replica r of
 * topology g).  DEVICE arrays:
 *   x_op  [R][n_op_total][f_op]    fp32
 *   x_dev [R][n_dev_total][f_dev]  fp32
 *   x_oo  replica r at x_oo + r*stride_oo, [E_oo]      fp32 (log tensor size)
 *   x_dd  replica r at x_dd + r*stride_dd, [E_dd][2]   fp32
 *   x_od  replica r at x_od + r*stride_od, [E_od]      uint8 placement bit
 *         (any nonzero value counts as 1)
 * A stride of 0 shares one copy among all replicas.  Strides are in elements.
 */
typedef struct tag_features {
    int32_t n_replicas;
    const float *x_op, *x_dev, *x_oo, *x_dd;
    const uint8_t *x_od;
    int64_t stride_oo, stride_dd, stride_od;
} tag_features;

/* Workspace bytes tag_gnn_forward needs for this graph, dims and R. */
tag_status tag_gnn_workspace(const tag_graph *g, const tag_model_dims *dims,
                             int32_t n_replicas, size_t *bytes);

/*
 * The forward pass of Section 4.2.1 for every candidate of the batch.
 * Per layer l, link type r, destination u and neighbour v:
 *   m_uv  = sigma(W^h h_v + W^e e_uv + b)       (ReLU, or ELU: dims->sigma)
 *   s_uvk = LeakyReLU(a^(k) . m_uv^(k) + adst^(k) . (W^h h_u)^(k))
 *   alpha = softmax of s over u's neighbours of link type r, per head
 *   h'_u  = sum_r gamma_r sum_v alpha_uv m_uv     (empty bucket: 0)
 * Outputs (DEVICE fp32): E_op [R][n_op_total][f], E_dev [R][n_dev_total][f].
 * Asynchronous on hip_stream; allocates nothing; workspace is scratch for
 * the duration of the call (calls that share a workspace must be ordered).
 */
tag_status tag_gnn_forward(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                           const tag_features *x, void *workspace, size_t ws_bytes,
                           float *E_op, float *E_dev, void *hip_stream);

/* ------------------------------------------------------------------------ */
/* Decision head                                                             */
/* ------------------------------------------------------------------------ */

/*
 * Strategy slice table (DEVICE): slice a places the op on the devices whose
 * bits are set in mask[a] (bit j = local device j of the query's topology;
 * bits at or above that topology's device count are ignored) with
 * replication option option[a]:
 *   0 replicate + AllReduce   1 replicate + parameter server
 *   2 duplicate (sufficient-factor broadcasting; no gradient sync)
 *   3 model parallel
 */
typedef struct tag_slices {
    int32_t n_slices;              /* S >= 1 */
    const uint64_t *mask;          /* DEVICE [S] */
    const uint8_t *option;         /* DEVICE [S], values 0..3 (others: treated as 3) */
} tag_slices;

/* Decoded decision for one query (the argmax slice). */
typedef struct tag_decision {
    uint64_t mask;        /* placement (bits of valid devices only)            */
    int32_t option;       /* 0..3 as above                                     */
    int32_t replicas;     /* popcount(mask) for options 0-2, 1 for option 3    */
    int32_t sync;         /* 0 AllReduce, 1 parameter server, 2 none           */
    int32_t sfb;          /* 1 if the compression (SFB, duplicate) option      */
} tag_decision;

tag_status tag_gnn_decide_workspace(const tag_graph *g, const tag_model_dims *dims,
                                    int32_t n_replicas, int32_t n_slices, int32_t n_query,
                                    size_t *bytes);

/*
 * Scores every slice for each query op (replica query_rep[q], topology
 * query_graph[q], local op query_op[q]):
 *   x     = [ sum_{j in mask} E_dev[j] ; E_op[i] ; onehot(option) ]
 *   score = w2 . ReLU(W1 x + b1) + b2     (H > 0)   or   w2 . x + b2  (H = 0)
 *   prior = softmax over the S slices, argmax = lowest index among maxima.
 * Outputs (DEVICE): argmax [Q] int32, best_score [Q] fp32, and optionally
 * prior [Q][S] fp32 and decision [Q] (either may be NULL).  Query indices
 * are DEVICE int32 arrays; out-of-range queries produce argmax -1, a NaN
 * score and an all-zero decision.  Asynchronous.
 */
tag_status tag_gnn_decide(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                          int32_t n_replicas, const float *E_op, const float *E_dev,
                          const tag_slices *slices, int32_t n_query, const int32_t *query_rep,
                          const int32_t *query_graph, const int32_t *query_op,
                          int32_t *argmax, float *best_score, float *prior, tag_decision *decision,
                          void *workspace, size_t ws_bytes, void *hip_stream);

/*
 * Allocation-free variant of tag_gnn_decide, for callers that cannot
 * allocate device memory or pass a workspace: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  Same arguments,
 * results and errors as tag_gnn_decide, without workspace/ws_bytes: the
 * scratch is a static device array inside the library of
 * tag_gnn_decide_noalloc_max_bytes() bytes (64 MiB), one copy per GPU,
 * held until the process ends; its address is looked up once per device
 * (on the device current at the first call).  A problem whose workspace
 * (tag_gnn_decide_workspace) exceeds that size is rejected with
 * TAG_ENOSPACE before anything is enqueued.  Every call on one GPU shares
 * that GPU's scratch: calls that overlap in time on one GPU (different
 * streams or host threads without ordering) race and must be serialised by
 * the caller.  Nothing in the scratch needs to start at zero: every value a
 * call reads was written earlier in the same call.  Asynchronous.
 */
size_t tag_gnn_decide_noalloc_max_bytes(void);
tag_status tag_gnn_decide_noalloc(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                                  int32_t n_replicas, const float *E_op, const float *E_dev,
                                  const tag_slices *slices, int32_t n_query, const int32_t *query_rep,
                                  const int32_t *query_graph, const int32_t *query_op,
                                  int32_t *argmax, float *best_score, float *prior, tag_decision *decision,
                                  void *hip_stream);

/*
 * Full-enumeration variant of tag_gnn_decide (topologies of at most 16
 * devices, dec_hidden <= 512): the slices are every non-empty device mask
 * of the query's topology with each option, slice a = 4 (mask - 1) + option
 * (bit j of mask = local device j), scored as tag_gnn_decide scores a slice
 * table.  Prior rows have S_full = 4 (2^max_dev - 1) entries (max_dev from
 * tag_graph_get_info); a query of a topology with fewer devices fills the
 * first 4 (2^n_dev - 1) and gets zeros after.  argmax = lowest slice index
 * among maxima; out-of-range queries as in tag_gnn_decide.  No slice table
 * is materialised: masks are walked in Gray-code order, one device row added
 * or removed per step.  Asynchronous.
 */
tag_status tag_gnn_decide_full_workspace(const tag_graph *g, const tag_model_dims *dims, int32_t n_replicas,
                                         int32_t n_query, size_t *bytes);
tag_status tag_gnn_decide_full(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                               int32_t n_replicas, const float *E_op, const float *E_dev, int32_t n_query,
                               const int32_t *query_rep, const int32_t *query_graph, const int32_t *query_op,
                               int32_t *argmax, float *best_score, float *prior, tag_decision *decision,
                               void *workspace, size_t ws_bytes, void *hip_stream);

/* Thread-local description of the last non-OK status ("" if none). */
const char *tag_last_error(void);

/* Library version string. */
const char *tag_version(void);

#ifdef __cplusplus
}
#endif
#endif /* TAG_H */
