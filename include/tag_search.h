/*
 * tag_search.h -- C ABI of the batched strategy-search service around the
 * GNN hot path: a PUCT tree search over per-group strategy slices whose
 * priors come from tag_gnn_forward + tag_gnn_decide in batches of leaves
 * (Section 4.2.2 of the paper, Monte-Carlo Tree Search).
 *
 * Pieces:
 *   tag_search_problem_*  the static problem: op groups, the slice table,
 *                         the analytic iteration-time model that gives the
 *                         reward, and the feature encoding of a search state
 *   tag_mcts_*            the search tree (host): PUCT selection, batched
 *                         with in-flight visits, expansion, back-propagation
 *   tag_search_pack       host: leaves -> rewards + compact state records
 *   tag_search_features   GPU: state records -> GNN inputs of the batch
 *
 * Readings of the paper (its text leaves these open):
 *  - Op groups are decided in descending order of total FLOPs (equal totals:
 *    lower group id first); tree depth d = the first d groups decided.
 *  - An action is a slice (device mask, replication option) of the slice
 *    table; the prior of slice a at a state is the decoder's softmax prior of
 *    the next group's representative op (its op with the most FLOPs, lower
 *    id on ties).
 *  - PUCT: U = Q + c G sqrt(sum N) / (1 + N); unvisited Q = 0; the first
 *    maximum wins.  Q is the running mean of the rewards seen through the
 *    edge: Q += (r - Q) / N.
 *  - Batching: B leaves are selected one after another; each edge on a
 *    selected path holds an in-flight visit counted with reward `vl_value`
 *    (N_eff = N + VL, Q_eff = (N Q + VL vl_value) / N_eff) until the round's
 *    update, which applies the leaves in selection order (expand if not yet
 *    expanded, then replace every in-flight visit by the real one).
 *  - Reward: the speed-up of the strategy's modelled iteration time over the
 *    baseline (every group on every device, AllReduce), or -1 when a device
 *    runs out of memory or a group's mask names no device.  Undecided groups
 *    take the strategy of the first decided group; with none decided, the
 *    baseline.  The model (per group g on devices D, r = |D|):
 *      compute on j in D: FLOPs_g / speed_j (duplicate) or / (r speed_j)
 *      communication:     AllReduce 2 (r-1)/r params_g / min bw(D);
 *                         PS 2 (r-1)/r params_g / min bw(first of D, D);
 *                         duplicate and model parallel (r-1)/r acts_g / min bw(D)
 *      device time = sum of compute + communication of its groups;
 *      iteration time = max device time + cross-group tensor bytes over the
 *      link between the groups' first devices (when their masks differ);
 *      memory on j = 4 params_g (divided by r for model parallel) +
 *      activations acts_g (divided by r unless duplicate).
 *    It stands in for the paper's simulator, which needs profiles of real
 *    training graphs.
 *
 * Memory: host handles are owned by the library (create/destroy).  Device
 * buffers are caller-owned; tag_search_device_bytes gives their sizes.
 * Errors follow tag.h (tag_status, tag_last_error()).
 */
#ifndef TAG_SEARCH_H
#define TAG_SEARCH_H

#include "tag.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tag_search_problem tag_search_problem;   /* opaque host handle */
typedef struct tag_mcts tag_mcts;                       /* opaque host handle */

/* Static inputs (HOST arrays, copied by tag_search_problem_create). */
typedef struct tag_search_problem_desc {
    int32_t n_op, n_dev, n_groups, n_slices;
    int32_t f_op;                            /* op feature width: 40 or 42      */
    const int32_t *group_of;                 /* [n_op] group of every op        */
    const int32_t *op_type;                  /* [n_op] op type (one-hot mod 32) */
    const double *op_flops;                  /* [n_op] FLOPs per iteration      */
    const double *op_bytes;                  /* [n_op] output tensor bytes      */
    const double *op_params;                 /* [n_op] parameter bytes          */
    const double *dev_tflops;                /* [n_dev]                         */
    const double *dev_mem_gb;                /* [n_dev]                         */
    const double *dev_intra_gbs;             /* [n_dev] bandwidth inside a device group */
    int64_t e_dd;
    const int32_t *dd_a, *dd_b;              /* [e_dd] unordered device links   */
    const double *dd_gbs;                    /* [e_dd] link bandwidth, GB/s     */
    int64_t e_oo;
    const int32_t *oo_src, *oo_dst;          /* [e_oo] tensors between ops      */
    int64_t e_od;
    const int32_t *od_op, *od_dev;           /* [e_od] op-device pairs in the   */
                                             /* order of the GNN's od features  */
    const uint64_t *slice_mask;              /* [n_slices] device masks         */
    const uint8_t *slice_option;             /* [n_slices] 0 AllReduce, 1 PS,   */
                                             /* 2 duplicate, 3 model parallel   */
} tag_search_problem_desc;

/* Validates and copies the problem: n_dev in [1, 64], n_groups >= 1, every
 * group id in range and used, positive FLOPs, speeds, memories and
 * bandwidths, every device pair linked (TAG_EINVAL / TAG_ERANGE otherwise),
 * f_op 40 or 42 (TAG_ESHAPE). */
tag_status tag_search_problem_create(const tag_search_problem_desc *desc, tag_search_problem **out);
void tag_search_problem_destroy(tag_search_problem *p);

/* The search order of the groups (descending FLOPs), order[i] = group decided
 * at depth i, and the representative op of every group. */
tag_status tag_search_order(const tag_search_problem *p, int32_t *order /*[n_groups]*/,
                            int32_t *rep_op /*[n_groups]*/);

/* Reward of the partial strategy `path[0..depth)` (slice ids of the first
 * `depth` groups in search order), with its modelled iteration time and OOM
 * flag.  depth in [0, n_groups], slice ids in [0, n_slices). */
tag_status tag_search_evaluate(const tag_search_problem *p, const int32_t *path, int32_t depth,
                               double *reward, double *iter_time, int32_t *oom);

/* Reward and runtime-feedback model: 0 (the default) the analytic model
 * above; 1 the simulator (tag_simulate below).  The model gives the reward
 * (baseline time over iteration time, recomputed for the baseline when the
 * model changes) and the runtime feedback that tag_search_pack writes into
 * the state records (op features: log10 of the group's makespan in ms and
 * its idle share; device features: memory share and idle share):
 *   analytic:  makespan = slowest replica's compute, idle share = sync /
 *              (compute + sync), memory = the modelled use, device idle =
 *              1 - load / time
 *   simulator: the simulated group makespan, group idle before its output
 *              transfers / iteration time, peak memory / capacity (both
 *              memory shares capped at 1) and device idle share, plus each
 *              link's idle share (tag_search_link_features).
 * TAG_EINVAL for another value or a tensor graph with a cycle (simulator). */
tag_status tag_search_set_model(tag_search_problem *p, int32_t model);

/* ---- search tree -------------------------------------------------------- */

/* n_levels = number of groups, n_actions = number of slices (<= 4096),
 * c_puct >= 0, vl_value finite.  The root (depth 0) starts unexpanded. */
tag_status tag_mcts_create(int32_t n_levels, int32_t n_actions, double c_puct, double vl_value,
                           tag_mcts **out);
void tag_mcts_destroy(tag_mcts *t);

/* Select B >= 1 leaves.  For leaf b: leaf[b] is its vertex id, depth[b] its
 * depth and path[b * n_levels + i] (i < depth[b]) the actions from the root.
 * Each edge on the path now holds one in-flight visit. */
tag_status tag_mcts_select(tag_mcts *t, int32_t B, int32_t *leaf, int32_t *depth, int32_t *path);

/* Apply the B leaves of an earlier select, in order: a leaf with depth <
 * n_levels that is not expanded yet is expanded with priors[b * n_actions +
 * a] (>= 0, finite); then every edge of its path gets reward rewards[b].
 * The arguments must be exactly those a select returned and that no update
 * has applied yet; several selects may be outstanding (TAG_EINVAL if a path
 * does not match the tree or holds no in-flight visit). */
tag_status tag_mcts_update(tag_mcts *t, int32_t B, const int32_t *leaf, const int32_t *depth,
                           const int32_t *path, const float *priors, const double *rewards);

/* Root edges: visit counts and mean rewards (n_actions each). */
tag_status tag_mcts_root_stats(const tag_mcts *t, int32_t *visits, double *q);

/* The most-visited path (first maximum per level), stopping at an unvisited
 * or unexpanded vertex; *depth receives its length. */
tag_status tag_mcts_best_path(const tag_mcts *t, int32_t *path, int32_t *depth);

/* Vertex count and expanded-vertex count. */
tag_status tag_mcts_size(const tag_mcts *t, int64_t *vertices, int64_t *expanded);

/* ---- batched evaluation of leaves on the GPU ---------------------------- */

/* Device buffer sizes: the static part (uploaded once) and one packed state
 * record per candidate. */
tag_status tag_search_device_bytes(const tag_search_problem *p, size_t *static_bytes,
                                   size_t *state_bytes);

/* Copy the static part (op attributes, device attributes, op-device pairs)
 * into the DEVICE buffer `static_dev` (synchronous). */
tag_status tag_search_upload(const tag_search_problem *p, void *static_dev, size_t bytes, void *hip_stream);

/* For the B leaves of a select: write their rewards, the query op of the
 * next group (its representative op; 0 for complete strategies) and one
 * packed state record each into HOST memory `states` (B * state_bytes).
 * Under the simulator model the leaves are simulated on up to 16 host
 * threads (results do not depend on the thread count). */
tag_status tag_search_pack(const tag_search_problem *p, int32_t B, const int32_t *depth,
                           const int32_t *path, int32_t path_stride, void *states, double *rewards,
                           int32_t *query_op);

/* GPU: expand the B packed records (DEVICE `states_dev`) into the GNN inputs
 * of the batch: x_op [B][n_op][f_op], x_dev [B][n_dev][8] (float32) and x_od
 * [B][e_od] (uint8), all DEVICE.  Asynchronous on hip_stream. */
tag_status tag_search_features(const tag_search_problem *p, int32_t B, const void *static_dev,
                               const void *states_dev, float *x_op, float *x_dev, uint8_t *x_od,
                               void *hip_stream);

/* GPU: the link rows of the B packed records, x_dd [B][e_dd][2] (float32,
 * DEVICE): log10(link GB/s) - 1 and the link's idle share (the simulator's;
 * 0 under the analytic model).  Asynchronous on hip_stream. */
tag_status tag_search_link_features(const tag_search_problem *p, int32_t B, const void *static_dev,
                                    const void *states_dev, float *x_dd, void *hip_stream);

/* ---- native search rounds ---------------------------------------------- */

/* Everything a run of search rounds needs.  The GNN inputs of a leaf are the
 * features tag_search_features writes plus the shared x_oo rows and x_dd
 * rows: the caller's shared rows under the analytic model, the leaf's own
 * (tag_search_link_features) under the simulator model. */
typedef struct tag_search_run_args {
    const tag_search_problem *problem;
    tag_mcts *tree;                   /* n_levels = n_groups, n_actions = n_slices       */
    const tag_graph *graph;           /* built from the problem's topology (one topology) */
    const tag_model_dims *dims;       /* f_op must equal the problem's f_op               */
    const tag_weights *weights;       /* DEVICE parameters                                */
    const float *x_oo;                /* DEVICE [e_oo] tensor features of every leaf      */
    const float *x_dd;                /* DEVICE [e_dd][2] link features (analytic model)  */
    const tag_slices *slices;         /* DEVICE copy of the problem's slice table         */
    int32_t batch;                    /* B >= 1 leaves per round                          */
    int32_t rounds;                   /* >= 1                                             */
    int32_t pipelined;                /* 1: round k+1 is selected, packed and enqueued    */
                                      /* before round k's update (its paths then also     */
                                      /* carry round k's in-flight visits); 0: strictly   */
                                      /* select, evaluate, update per round               */
    void *workspace;                  /* DEVICE, >= tag_search_run_workspace dev_bytes   */
    size_t ws_bytes;
    void *host_buf;                   /* pinned HOST, >= host_bytes                       */
    size_t host_bytes;
    /* optional HOST outputs (NULL to skip), in selection order:                          */
    int32_t *depth_out;               /* [rounds * B]                                     */
    int32_t *path_out;                /* [rounds * B * n_groups]                          */
    double *reward_out;               /* [rounds * B]                                     */
    float *prior_out;                 /* [rounds * B * n_slices]                          */
} tag_search_run_args;

tag_status tag_search_run_workspace(const tag_search_problem *p, const tag_graph *g, const tag_model_dims *dims,
                                    int32_t batch, size_t *dev_bytes, size_t *host_bytes);

/* Run `rounds` rounds: select B leaves, compute their rewards and states on
 * the host, expand the states, forward + decide on the GPU (one query per
 * leaf: the next group's representative op), update the tree with the
 * priors and rewards.  Synchronous: returns when the last update is done.
 * Uses only the caller's buffers (no allocation on the device).  On a
 * non-OK status the stream has been drained, and the tree may still hold
 * the in-flight visits of rounds that were selected but not updated. */
tag_status tag_search_run(const tag_search_run_args *a, void *hip_stream);

/* ---- simulator (Section 4.3.2, with the auxiliary ops of Section 4.3.1) -- */

/*
 * Simulates one training iteration of a strategy and reports the runtime
 * feedback the GNN takes as input (Section 4.2.1: group makespan, idle time
 * before a group's output transfers, device peak memory and idle share,
 * link idle share).  Readings of the paper:
 *  - Every op takes its group's device set D (r = |D|) and option.  Compute
 *    task per device j of D: FLOPs / speed_j (duplicate or r = 1), else
 *    FLOPs / (r speed_j).
 *  - Model parallel, r > 1: a gather task per device after all partitions,
 *    (r - 1) / r out_bytes / min bandwidth inside D; consumers read its output.
 *  - Options 0 / 1, r > 1, parameters > 0: a sync task per device after all
 *    replicas, 2 (r - 1) / r params / (min bandwidth inside D for AllReduce,
 *    min bandwidth from D's first device for the parameter server).
 *  - Tensor p -> c, device j of c: local when j holds p; else a transfer
 *    from p's device with the highest bandwidth to j (first maximum) on that
 *    link, out_bytes(p) / r_c bytes when c splits its batch (options 0, 1),
 *    the whole tensor otherwise, taking bytes / bandwidth.
 *  - One FIFO queue per device and per device pair.  Tasks are numbered per
 *    op (compute tasks in device order, gathers, syncs), then per tensor in
 *    input order (transfers in device order); completions are processed by
 *    (finish time, task number), the tasks they make ready enter their
 *    queues in task-number order, an idle resource starts at once.
 *  - Memory: 4 x parameters resident on every device of D (divided by r for
 *    model parallel); a task's output (compute: out_bytes, or out_bytes / r
 *    when split; gather: out_bytes; transfer: its bytes) is allocated when
 *    it finishes, then its inputs are released; a tensor is freed after its
 *    last use (a tensor without uses at once).
 *  - Outputs: iteration time = last finish; group makespan = last finish of
 *    its compute / gather / sync tasks - first start of its compute tasks;
 *    group idle = mean over transfers to another group's op of transfer
 *    start - producer finish (0 without); idle share = 1 - busy / time; OOM
 *    when a peak exceeds the device memory.
 * It needs no GPU.
 */
typedef struct tag_sim_out {
    double iter_time;          /* seconds; +inf for an invalid strategy          */
    int32_t valid;             /* 0: a group's device set is empty               */
    int32_t oom;               /* 1 when out of memory (or invalid)              */
    int64_t n_tasks;
    double *group_makespan;    /* HOST [n_groups] seconds, or NULL               */
    double *group_idle;        /* HOST [n_groups] seconds, or NULL               */
    double *dev_peak;          /* HOST [n_dev] bytes, or NULL                    */
    double *dev_idle;          /* HOST [n_dev] share of the iteration, or NULL   */
    double *link_idle;         /* HOST [e_dd] share, links in input order, or NULL */
} tag_sim_out;

/* Simulate the strategy path[0..depth) completed as in tag_search_evaluate.
 * TAG_EINVAL if the tensor graph has a cycle. */
tag_status tag_simulate(const tag_search_problem *p, const int32_t *path, int32_t depth, tag_sim_out *out);

/* B strategies (depth[b], path + b * path_stride) on n_threads host threads
 * (1..256): iteration times and OOM flags (HOST arrays [B]). */
tag_status tag_simulate_batch(const tag_search_problem *p, int32_t B, const int32_t *depth, const int32_t *path,
                              int32_t path_stride, int32_t n_threads, double *iter_time, int32_t *oom);

#ifdef __cplusplus
}
#endif

#endif /* TAG_SEARCH_H */
