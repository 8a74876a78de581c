/*
 * tag_train.h -- C ABI of the GNN training step: the cross entropy between
 * the decoder's priors and target distributions over the strategy slices
 * (the search's selection probabilities), its gradient with respect to every
 * parameter, and an optional SGD update (Section 4.2.2: the GNN parameters
 * are updated to minimise the cross entropy between the prior G(s, a) and the
 * MCTS selection probability pi(s, a)).
 *
 *   loss = -(1/Q) sum_q sum_a target[q][a] log prior[q][a]
 *
 * prior[q] is tag_gnn_decide's softmax for query q (replica query_rep[q],
 * topology query_graph[q], local op query_op[q]) of the same forward pass
 * tag_gnn_forward computes.  The gradient flows through the decoder, every
 * GAT layer (messages, attention logits, the per-destination softmax, the
 * gamma-weighted sums, the relation transforms and the folded edge encoders)
 * and the node encoders.
 *
 * Scope: fp32 models (dims->dtype TAG_F32; ReLU or ELU messages) with the MLP decoder
 * (dec_hidden >= 1) and at most 4096 slices; TAG_ESHAPE otherwise.  A query
 * whose indices are out of range contributes nothing (its loss term and
 * gradient are zero; Q still counts it).  Every reduction runs in a fixed
 * order, so a step is bitwise repeatable.  Conventions follow tag.h:
 * caller-owned DEVICE buffers, asynchronous on hip_stream, no allocation.
 */
#ifndef TAG_TRAIN_H
#define TAG_TRAIN_H

#include "tag.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Gradient arrays: DEVICE float32, the same shapes as the matching
 * parameters of tag_weights (enc_op_w [f][f_op], ..., layer_w [L][3][f][2f],
 * ..., dec_w1 [H][2f+4], dec_b1 [H], dec_w2 [H], dec_b2 [1]).  Overwritten. */
typedef struct tag_grads {
    float *enc_op_w, *enc_op_b, *enc_dev_w, *enc_dev_b;
    float *enc_edge_w[3], *enc_edge_b[3];
    float *layer_w, *layer_b, *att_src, *att_dst;
    float *dec_w1, *dec_b1, *dec_w2, *dec_b2;
} tag_grads;

/* Targets: DEVICE arrays, Q queries of the batch. */
typedef struct tag_train_batch {
    int32_t n_query;                 /* Q >= 1                                   */
    const int32_t *query_rep;        /* [Q] replica of each query                */
    const int32_t *query_graph;      /* [Q] topology of each query               */
    const int32_t *query_op;         /* [Q] op (local id in its topology)        */
    const float *target;             /* [Q][S] target distribution of each query  */
} tag_train_batch;

tag_status tag_train_workspace(const tag_graph *g, const tag_model_dims *dims, int32_t n_replicas,
                               int32_t n_slices, int32_t n_query, size_t *bytes);

/* One training step over the n_replicas candidates of `x`: forward pass,
 * loss (DEVICE float [1]), gradients (`grad`, overwritten) and, when
 * lr > 0, the update w -= lr * grad applied in place to the DEVICE
 * parameter arrays of `w` (which must then be writable; the gradients are
 * those of the parameters before the update).  The workspace holds every
 * layer's saved activations, the backward buffers and the per-query
 * partials (tag_train_workspace gives its size). */
tag_status tag_train_step(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                          const tag_features *x, const tag_slices *slices, const tag_train_batch *batch,
                          const tag_grads *grad, float lr, float *loss, void *workspace, size_t ws_bytes,
                          void *hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* TAG_TRAIN_H */
