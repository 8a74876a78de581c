// Forward-pass internals shared with the training step (train.hip).
#pragma once

#include "agg_common.hpp"

namespace tag {

// Workspace layout of tag_gnn_forward.
struct FwdLayout {
    float *U, *cp;                 // folded edge terms per (layer, relation)
    uint16_t *Wb;                  // bf16 copies of W^h (bf16 variant)
    void *H_op[2], *H_dev[2];      // ping-pong hidden rows
    void *Y_op, *Y_dev;            // [R*n][2F] relation transforms (+ folded bias)
    float *part;
    int32_t maxc;
    bool mfma;
    uint64_t *omask;
    float *Sdev, *T, *Sop;
    int32_t *tile_ext;             // per op tile descriptors (see AggArgs)
    float *xcsr;                   // op<-op edge features in CSR order
};

tag_status check_dims(const tag_model_dims *d);

// The readings of variants.hip (five directed relations, ReLU edge
// encoders, averaged full-width heads): generic fp32 forward path.
bool is_variant(const tag_model_dims *d);
tag_status check_variant(const tag_model_dims *d);
size_t variant_workspace(const tag_graph *g, const tag_model_dims *d, int32_t R);
tag_status forward_variant(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                           const tag_features *x, void *workspace, size_t ws_bytes, float *E_op, float *E_dev,
                           hipStream_t stream);
size_t carve_fwd(const tag_graph *g, const tag_model_dims *d, int32_t R, void *base, FwdLayout *L);

// Where a forward pass keeps every layer's activations (fp32): the input
// rows H^l of layer l = 0 .. L-1 go to H_op[l] / H_dev[l] and its relation
// transforms (stored as W^h h + c', [rows][2f]) to Y_op[l] / Y_dev[l]; the
// last layer writes E_op / E_dev.
struct FwdSave {
    float *H_op[16], *H_dev[16];
    float *Y_op[16], *Y_dev[16];
};

tag_status forward_run(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w, const tag_features *x,
                       void *workspace, size_t ws_bytes, float *E_op, float *E_dev, hipStream_t stream,
                       const FwdSave *save);
void launch_layer_transform(const tag_graph *g, const tag_model_dims *dims, const tag_weights *w,
                            const FwdLayout &L, int32_t R, int l, const void *H_op, const void *H_dev,
                            hipStream_t stream);

}  // namespace tag
