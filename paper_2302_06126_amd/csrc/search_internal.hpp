// Internal declarations of the strategy-search service (search_host.hip,
// search_features.hip).
#pragma once

#include <algorithm>
#include <vector>

#include "tag_internal.hpp"
#include "../../include/tag_search.h"

struct tag_search_problem {
    int32_t N = 0, M = 0, K = 0, S = 0, f_op = 42;
    std::vector<int32_t> group_of, op_type;
    std::vector<double> op_flops, op_bytes;
    std::vector<double> FL, PB, AB;          // per group: FLOPs, parameter bytes, activation bytes
    std::vector<int32_t> order, rep;         // search order of the groups; representative op per group
    std::vector<double> speed, mem;          // per device: flop/s, bytes
    std::vector<double> dev_tflops, dev_mem_gb, dev_intra;
    std::vector<double> bw;                  // [M][M] bytes/s (diagonal: inside the device group)
    std::vector<std::pair<int, int>> xpairs; // cross-group tensor traffic, first-appearance order
    std::vector<double> xbytes;
    std::vector<int32_t> od_op, od_dev;
    std::vector<double> op_params;           // per op (the simulator works per op)
    std::vector<int32_t> oo_src, oo_dst;     // tensors in input order
    std::vector<int32_t> dd_a, dd_b;         // device links in input order
    std::vector<double> dd_gbs;              // their bandwidths, GB/s
    std::vector<uint64_t> slice_mask;
    std::vector<int32_t> slice_opt;
    double T_base = 0.0;                     // baseline iteration time
    int32_t model = 0;                       // 0 analytic model, 1 simulator
};

namespace tag {

struct Eval {
    double T = 0.0;
    bool oom = false;
    std::vector<double> load, mem, comp, sync;
};

void full_strategy(const tag_search_problem *P, const int32_t *path, int32_t depth, uint64_t *mask, int32_t *opt);
Eval evaluate_strategy(const tag_search_problem *P, const uint64_t *mask, const int32_t *opt);

// Simulator (simulate.hip).  Scratch reused across simulations of one
// thread.  Returns false when the tensor graph has a cycle.
struct SimScratch;
SimScratch *sim_scratch_new();
void sim_scratch_free(SimScratch *w);
bool sim_run(const tag_search_problem *P, const uint64_t *mask, const int32_t *opt, SimScratch *W, double *T,
             bool *valid, bool *oom, double *g_makespan, double *g_idle, double *d_peak, double *d_idle,
             double *l_idle);

// Host threads tag_search_pack uses under the simulator model.
constexpr int kPackThreads = 16;

// Runtime feedback of a full strategy under the problem's model (search_host.hip).
struct Feedback {
    double T = 0.0;
    bool oom = false;
    std::vector<double> gms, gidle, memf, didle, peak, lidle;
};
bool strategy_feedback(const tag_search_problem *P, const uint64_t *mask, const int32_t *opt, SimScratch *W,
                       Feedback *f);

// Static device part: group_of, op_type [N] int32; lflops, lbytes [N] float;
// device rows [M][4] float; od_op, od_dev [E_od] int32; link rows
// log10(GB/s) - 1 [E_dd] float.
struct StaticLayout {
    size_t group_of, op_type, lflops, lbytes, dev, od_op, od_dev, dd_lbw, total;
};
inline StaticLayout static_layout(const tag_search_problem *p) {
    StaticLayout s;
    size_t o = 0;
    auto take = [&](size_t bytes) { const size_t r = o; o = align_up(o + bytes, 16); return r; };
    s.group_of = take(4 * (size_t)p->N);
    s.op_type = take(4 * (size_t)p->N);
    s.lflops = take(4 * (size_t)p->N);
    s.lbytes = take(4 * (size_t)p->N);
    s.dev = take(16 * (size_t)p->M);
    s.od_op = take(4 * p->od_op.size());
    s.od_dev = take(4 * p->od_op.size());
    s.dd_lbw = take(4 * p->dd_a.size());
    s.total = std::max<size_t>(o, 16);
    return s;
}

// One packed state record: int32 next group (-1: complete), int32 pad;
// uint64 mask[K]; int32 option[K]; int32 decided[K]; float gfeat[K][2]
// (log10 makespan ms, idle fraction of decided groups); float dfeat[M][2]
// (peak-memory fraction, idle fraction); float lfeat[E_dd] (link idle
// share: the simulator's, 0 under the analytic model).
struct StateLayout {
    size_t mask, option, decided, gfeat, dfeat, lfeat, total;
};
inline StateLayout state_layout(const tag_search_problem *p) {
    StateLayout s;
    const size_t K = p->K, M = p->M;
    s.mask = 8;
    s.option = s.mask + 8 * K;
    s.decided = s.option + 4 * K;
    s.gfeat = s.decided + 4 * K;
    s.dfeat = s.gfeat + 8 * K;
    s.lfeat = s.dfeat + 8 * M;
    s.total = align_up(s.lfeat + 4 * p->dd_a.size(), 16);
    return s;
}

}  // namespace tag
