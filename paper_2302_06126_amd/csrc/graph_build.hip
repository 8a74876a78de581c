// Relation-bucketed CSR builder for the joint op/device graph.
//
// Section 4.2.1 of the paper defines the GNN input as a heterogeneous graph
// with two node types (op groups, device groups) and three link types
// (op-op tensors, device-device network links, op-device placements).  The
// layer aggregates, for each destination node, over its neighbours of each
// link type, so the graph is stored as four destination-keyed buckets:
//   B0 op<-op (both directions of every tensor link), B1 op<-dev,
//   B2 dev<-op, B3 dev<-dev (both directions of every network link).
// Entries of a row are ordered by (source id, edge id), which makes the
// result a deterministic function of the input link sets.
//
// Pipeline (all on the caller's stream, seven kernels): clear counters;
// count per-row degrees while validating ids (device rows counted in LDS
// first, since few device rows receive many links); exclusive scans to row
// pointers; clear cursors; scatter (arbitrary order inside a row); exact
// per-row rank sort of short rows; LDS-bitmap counting sort of long rows.
// The sorts also detect repeated (row, source) pairs.  One stream sync at
// the end reads the validation flags and per-bucket maximum degrees.
#include <algorithm>

#include "tag_internal.hpp"

namespace tag {

static thread_local std::string g_last_error;
void set_error(const std::string &msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }

tag_status launch_status(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) TAG_FAIL(TAG_EHIP, std::string(what) + ": " + hipGetErrorString(e));
    return TAG_OK;
}

namespace {

constexpr int kThreads = 256;
constexpr int kScanItems = 4;                       // per thread
constexpr int kScanTile = kThreads * kScanItems;    // per block
constexpr int kSmallScan = 1 << 16;                 // arrays up to this length: one block per bucket
constexpr int kPrivRows = 4096;                     // device rows counted in LDS when the total fits
constexpr int kShortRow = 64;                       // rows up to this length: one wavefront per row
constexpr int kBitmapRange = 14336;                 // source-id range sorted through an LDS bitmap (<= 60 KB)

// flags after the counters in the tmp buffer
enum { FLAG_RANGE = 0, FLAG_DUP = 1, FLAG_MAXDEG = 4 /* 4 entries */, FLAG_COUNT = 8 };

__global__ void fill_i32(int32_t *p, int64_t n, int32_t v) {
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

// topology owning entry i of a prefix-offset array off[0..G]
template <typename T>
__device__ __forceinline__ int32_t owner(const T *off, int32_t G, int64_t i) {
    int32_t lo = 0, hi = G;   // find last g with off[g] <= i
    while (hi - lo > 1) {
        int32_t mid = (lo + hi) >> 1;
        if (off[mid] <= i) lo = mid; else hi = mid;
    }
    return lo;
}

struct Buckets {
    int64_t rows[4], nnz[4];
    int32_t *cnt[4];
    int32_t *rp[4];
    int32_t *tcol[4], *teid[4], *rowof[4];
    int32_t *col[4], *eid[4];
};

struct Rel {                   // one link type
    const int32_t *a, *b;      // endpoints (local ids)
    const int64_t *off;        // link prefix offsets [G+1]
    const int32_t *a_off, *b_off;   // node prefix offsets of a's and b's type [G+1]
    int64_t n;
    int32_t same_type;         // self links rejected
    int32_t bk_ba, bk_ab;      // bucket fed as (row = b, col = a) and as (row = a, col = b)
    int32_t priv_ba, priv_ab;  // that side's rows are device rows counted in LDS
};

struct EdgeArgs {
    Rel rel[3];
    int64_t blk_off[4];        // block ranges of the three relations
    int32_t G;
    int32_t n_dev;             // total device rows (LDS counter range)
    Buckets B;
    int32_t *flags;
    int32_t *oo_head;          // [E_oo] consumer (global op id) of each tensor link
};

// MODE 0: count degrees; MODE 1: scatter entries.  One thread per link.
template <int MODE>
__global__ void __launch_bounds__(kThreads) edges_pass(EdgeArgs A) {
    __shared__ int32_t lcnt[kPrivRows];
    __shared__ int32_t lbase[kPrivRows];
    const int64_t bid = blockIdx.x;
    const int r = bid < A.blk_off[1] ? 0 : (bid < A.blk_off[2] ? 1 : 2);
    const Rel R = r == 0 ? A.rel[0] : (r == 1 ? A.rel[1] : A.rel[2]);
    const bool priv = R.priv_ba || R.priv_ab;
    if (priv) {
        for (int i = threadIdx.x; i < A.n_dev; i += blockDim.x) lcnt[i] = 0;
        __syncthreads();
    }
    const int64_t i = (bid - A.blk_off[r]) * kThreads + threadIdx.x;
    bool ok = i < R.n;
    int32_t ga = 0, gb = 0;
    if (ok) {
        const int32_t g = owner(R.off, A.G, i);
        const int32_t la = R.a[i], lb = R.b[i];
        const int32_t na = R.a_off[g + 1] - R.a_off[g], nb = R.b_off[g + 1] - R.b_off[g];
        if (la < 0 || la >= na || lb < 0 || lb >= nb) {
            if (MODE == 0) atomicOr(&A.flags[FLAG_RANGE], 1);
            ok = false;
        } else if (R.same_type && la == lb) {
            if (MODE == 0) atomicOr(&A.flags[FLAG_DUP], 1);
            ok = false;
        } else {
            ga = R.a_off[g] + la;
            gb = R.b_off[g] + lb;
        }
    }
    // (row, col) of the two entries this link feeds
    const int32_t row0 = gb, col0 = ga, bk0 = R.bk_ba, row1 = ga, col1 = gb, bk1 = R.bk_ab;
    int32_t slot0 = 0, slot1 = 0;
    if (ok) {
        if (R.priv_ba) slot0 = atomicAdd(&lcnt[row0], 1);
        else slot0 = atomicAdd(&A.B.cnt[bk0][row0], 1);
        if (R.priv_ab) slot1 = atomicAdd(&lcnt[row1], 1);
        else slot1 = atomicAdd(&A.B.cnt[bk1][row1], 1);
    }
    if (priv) {
        // flush the LDS counters (both private sides of a relation share one bucket)
        __syncthreads();
        const int pb = R.priv_ba ? bk0 : bk1;
        for (int d = threadIdx.x; d < A.n_dev; d += blockDim.x) {
            const int32_t c = lcnt[d];
            if (c) {
                const int32_t base = atomicAdd(&A.B.cnt[pb][d], c);
                if (MODE == 1) lbase[d] = base;
            }
        }
        __syncthreads();
        if (MODE == 1 && ok) {
            if (R.priv_ba) slot0 += lbase[row0];
            if (R.priv_ab) slot1 += lbase[row1];
        }
    }
    if (MODE == 1 && ok) {
        if (r == 0) A.oo_head[i] = gb;   // the direction of each op<-op entry follows from it
        const int32_t p = A.B.rp[bk0][row0] + slot0;
        A.B.tcol[bk0][p] = col0; A.B.teid[bk0][p] = (int32_t)i; A.B.rowof[bk0][p] = row0;
        const int32_t q = A.B.rp[bk1][row1] + slot1;
        A.B.tcol[bk1][q] = col1; A.B.teid[bk1][q] = (int32_t)i; A.B.rowof[bk1][q] = row1;
    }
}

// ---- exclusive scans of int32 counts (n + 1 outputs, out[n] = total) ----
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, int32_t *total, int32_t *sh) {
    int tid = threadIdx.x;
    sh[tid] = v;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
        int32_t t = tid >= off ? sh[tid - off] : 0;
        __syncthreads();
        sh[tid] += t;
        __syncthreads();
    }
    int32_t incl = sh[tid];
    *total = sh[kThreads - 1];
    __syncthreads();
    return incl - v;
}

// one block per bucket, looping over tiles with a carry (moderate sizes)
__global__ void __launch_bounds__(kThreads) scan_buckets(Buckets B) {
    __shared__ int32_t sh[kThreads];
    const int b = blockIdx.x;
    const int64_t n = B.rows[b] + 1;
    int32_t carry = 0;
    for (int64_t base = 0; base < n; base += kScanTile) {
        const int64_t i0 = base + threadIdx.x * kScanItems;
        int32_t v[kScanItems], s = 0;
        for (int k = 0; k < kScanItems; ++k) {
            v[k] = (i0 + k < n) ? B.cnt[b][i0 + k] : 0;
            s += v[k];
        }
        // the counters restart at zero for the placement pass
        for (int k = 0; k < kScanItems; ++k)
            if (i0 + k < n) B.cnt[b][i0 + k] = 0;
        int32_t tot;
        int32_t ex = block_exclusive_scan(s, &tot, sh) + carry;
        for (int k = 0; k < kScanItems; ++k) {
            if (i0 + k < n) B.rp[b][i0 + k] = ex;
            ex += v[k];
        }
        carry += tot;
    }
}

__global__ void scan_tiles(const int32_t *in, int64_t n, int32_t *out, int32_t *tile_sums) {
    __shared__ int32_t sh[kThreads];
    int64_t base = (int64_t)blockIdx.x * kScanTile + threadIdx.x * kScanItems;
    int32_t v[kScanItems], s = 0;
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = (base + k < n) ? in[base + k] : 0;
        s += v[k];
    }
    int32_t tot;
    int32_t ex = block_exclusive_scan(s, &tot, sh);
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) out[base + k] = ex;
        ex += v[k];
    }
    if (threadIdx.x == 0) tile_sums[blockIdx.x] = tot;
}

// one block: exclusive scan of the tile sums in place, total to *grand
__global__ void scan_sums(int32_t *sums, int64_t n, int32_t *grand) {
    __shared__ int32_t sh[kThreads];
    int32_t carry = 0;
    for (int64_t base = 0; base < n; base += kThreads) {
        int64_t i = base + threadIdx.x;
        int32_t v = i < n ? sums[i] : 0;
        int32_t tot;
        int32_t ex = block_exclusive_scan(v, &tot, sh);
        if (i < n) sums[i] = ex + carry;
        carry += tot;
    }
    if (threadIdx.x == 0) *grand = carry;
}

__global__ void scan_add(int32_t *out, int64_t n, const int32_t *tile_sums) {
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i < n) out[i] += tile_sums[i / kScanTile];
}

// ---- exact per-row rank sort of short rows, all buckets in one launch ----
// One wavefront per row: lane i holds entry i of a row of at most 64
// entries, and its rank is counted against the others through lane
// shuffles.  Only the rp[rows] entries of a bucket were scattered (links
// rejected during the count pass never were).
__device__ void rank_rows(const Buckets &B, int64_t r1, int64_t r2, int64_t r3, int64_t rtot, int32_t *flags,
                          int64_t blk) {
    __shared__ int32_t bmax[4];
    if (threadIdx.x < 4) bmax[threadIdx.x] = 0;
    __syncthreads();
    const int64_t w = blk * (blockDim.x / 64) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (w < rtot) {
        const int b = w < r1 ? 0 : (w < r2 ? 1 : (w < r3 ? 2 : 3));
        const int64_t r = w - (b == 0 ? 0 : (b == 1 ? r1 : (b == 2 ? r2 : r3)));
        const int32_t beg = B.rp[b][r], end = B.rp[b][r + 1];
        const int32_t deg = end - beg;
        // rows of op<-dev and dev<-dev hold distinct devices of one topology
        // (at most 64): a longer row can only come from repeated pairs
        if ((b == 1 || b == 3) && deg > kShortRow && lane == 0) atomicOr(&flags[FLAG_DUP], 1);
        if (deg > 0 && deg <= kShortRow) {
            const bool mine = lane < deg;
            const int32_t c = mine ? B.tcol[b][beg + lane] : INT32_MAX;
            const int32_t e = mine ? B.teid[b][beg + lane] : INT32_MAX;
            int32_t rank = 0, dup = 0;
            for (int q = 0; q < deg; ++q) {
                const int32_t cq = __shfl(c, q, 64), eq = __shfl(e, q, 64);
                rank += (cq < c) || (cq == c && eq < e);
                dup |= (cq == c) && (q != lane);
            }
            if (mine) {
                B.col[b][beg + rank] = c;
                B.eid[b][beg + rank] = e;
                if (dup) atomicOr(&flags[FLAG_DUP], 1);
            }
            if (lane == 0) atomicMax(&bmax[b], deg);
        }
    }
    __syncthreads();
    if (threadIdx.x < 4 && bmax[threadIdx.x] > 0) atomicMax(&flags[FLAG_MAXDEG + threadIdx.x], bmax[threadIdx.x]);
}

// One block per row of B0 (blocks [0, rows0)) or B2 (the rest); only rows
// longer than kShortRow do work.  Sources of a row all belong to the row's
// topology, so a bitmap over that topology's source-id range sorts the row
// by source id (sources are unique in a valid row; a repeated source is
// caught by the atomic OR).  Ranges beyond the LDS bitmap (rmax source ids,
// at most kBitmapRange) fall back to the per-entry rank inside the block.
__device__ void rank_long_rows(const Buckets &B, const int32_t *op_off, const int32_t *dev_off, int32_t G,
                               int32_t rmax, int32_t *flags, int64_t blk) {
    extern __shared__ int32_t dyn[];   // bm [rmax/32] | wpre [rmax/32] | eid_of [rmax]
    __shared__ int32_t scan[256];
    const int nwmax = (rmax + 31) / 32;
    uint32_t *bm = reinterpret_cast<uint32_t *>(dyn);
    int32_t *wpre = dyn + nwmax;
    int32_t *eid_of = dyn + 2 * nwmax;
    const int b = blk < B.rows[0] ? 0 : 2;
    const int32_t r = b == 0 ? (int32_t)blk : (int32_t)(blk - B.rows[0]);
    const int32_t *rp = B.rp[b];
    const int32_t *tcol = B.tcol[b], *teid = B.teid[b];
    int32_t *col = B.col[b], *eid = B.eid[b];
    const int32_t beg = rp[r], end = rp[r + 1];
    if (end - beg <= kShortRow) return;
    const int32_t *row_off = b == 0 ? op_off : dev_off;
    const int32_t g = owner(row_off, G, r);
    const int32_t base = op_off[g], range = op_off[g + 1] - base;   // sources are ops in both buckets
    if (threadIdx.x == 0) atomicMax(&flags[FLAG_MAXDEG + b], end - beg);
    if (range > rmax) {
        for (int32_t p = beg + threadIdx.x; p < end; p += blockDim.x) {
            const int32_t c = tcol[p], e = teid[p];
            int32_t rank = 0, dup = 0;
            for (int32_t q = beg; q < end; ++q) {
                const int32_t cq = tcol[q], eq = teid[q];
                rank += (cq < c) || (cq == c && eq < e);
                dup |= (cq == c) && (q != p);
            }
            col[beg + rank] = c;
            eid[beg + rank] = e;
            if (dup) atomicOr(&flags[FLAG_DUP], 1);
        }
        return;
    }
    const int nw = (range + 31) / 32;
    for (int w = threadIdx.x; w < nw; w += blockDim.x) bm[w] = 0u;
    __syncthreads();
    int dup = 0;
    for (int32_t p = beg + threadIdx.x; p < end; p += blockDim.x) {
        const int32_t c = tcol[p] - base;
        const uint32_t bit = 1u << (c & 31);
        const uint32_t old = atomicOr(&bm[c >> 5], bit);
        dup |= (old & bit) != 0u;
        eid_of[c] = teid[p];
    }
    if (dup) atomicOr(&flags[FLAG_DUP], 1);
    __syncthreads();
    // exclusive prefix of per-word popcounts (chunks of 256 words)
    int32_t carry = 0;
    for (int w0 = 0; w0 < nw; w0 += 256) {
        const int w = w0 + threadIdx.x;
        const int32_t v = w < nw ? __popc(bm[w]) : 0;
        scan[threadIdx.x] = v;
        __syncthreads();
        for (int off = 1; off < 256; off <<= 1) {
            const int32_t t = threadIdx.x >= off ? scan[threadIdx.x - off] : 0;
            __syncthreads();
            scan[threadIdx.x] += t;
            __syncthreads();
        }
        if (w < nw) wpre[w] = carry + scan[threadIdx.x] - v;
        carry += scan[255];
        __syncthreads();
    }
    for (int w = threadIdx.x; w < nw; w += blockDim.x) {
        uint32_t bits = bm[w];
        int32_t pos = beg + wpre[w];
        while (bits) {
            const int k = __ffs(bits) - 1;
            bits &= bits - 1u;
            const int32_t c = w * 32 + k;
            col[pos] = base + c;
            eid[pos] = eid_of[c];
            ++pos;
        }
    }
}

// Both ranks in one launch: blocks [0, n_short) take four short rows each,
// the rest one B0 or B2 row each (long rows only).
__global__ void __launch_bounds__(256) rank_all(Buckets B, int64_t r1, int64_t r2, int64_t r3, int64_t rtot,
                                                int64_t n_short, const int32_t *op_off, const int32_t *dev_off,
                                                int32_t G, int32_t rmax, int32_t *flags) {
    if ((int64_t)blockIdx.x < n_short) rank_rows(B, r1, r2, r3, rtot, flags, blockIdx.x);
    else rank_long_rows(B, op_off, dev_off, G, rmax, flags, (int64_t)blockIdx.x - n_short);
}

inline unsigned grid_for(int64_t n, int64_t cap = 65536) {
    int64_t b = (n + kThreads - 1) / kThreads;
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>(b, cap));
}

struct Sizes {
    int32_t G = 0, max_dev = 0;
    int64_t n_op = 0, n_dev = 0, e_oo = 0, e_dd = 0, e_od = 0;
    int64_t rows[4], nnz[4];
};

tag_status check_desc(const tag_graph_desc *d, Sizes *s) {
    if (!d) TAG_FAIL(TAG_EINVAL, "graph descriptor is NULL");
    if (d->n_graphs < 1) TAG_FAIL(TAG_EINVAL, "n_graphs must be >= 1");
    if (!d->n_op || !d->n_dev || !d->oo_off || !d->dd_off || !d->od_off)
        TAG_FAIL(TAG_EINVAL, "n_op, n_dev and the three offset arrays must be non-NULL host arrays");
    s->G = d->n_graphs;
    const int64_t *offs[3] = {d->oo_off, d->dd_off, d->od_off};
    const char *names[3] = {"oo_off", "dd_off", "od_off"};
    for (int k = 0; k < 3; ++k) {
        if (offs[k][0] != 0) TAG_FAIL(TAG_EINVAL, std::string(names[k]) + "[0] must be 0");
        for (int32_t g = 0; g < d->n_graphs; ++g)
            if (offs[k][g + 1] < offs[k][g])
                TAG_FAIL(TAG_EINVAL, std::string(names[k]) + " must be non-decreasing");
    }
    for (int32_t g = 0; g < d->n_graphs; ++g) {
        if (d->n_op[g] < 1) TAG_FAIL(TAG_EINVAL, "every topology needs at least one op");
        if (d->n_dev[g] < 1) TAG_FAIL(TAG_EINVAL, "every topology needs at least one device");
        if (d->n_dev[g] > 64) TAG_FAIL(TAG_ESHAPE, "at most 64 devices per topology (slice masks are 64-bit)");
        s->n_op += d->n_op[g];
        s->n_dev += d->n_dev[g];
        s->max_dev = std::max(s->max_dev, d->n_dev[g]);
    }
    s->e_oo = d->oo_off[d->n_graphs];
    s->e_dd = d->dd_off[d->n_graphs];
    s->e_od = d->od_off[d->n_graphs];
    const int64_t lim = INT32_MAX - 1;
    if (s->n_op > lim || s->n_dev > lim || 2 * s->e_oo > lim || 2 * s->e_dd > lim || s->e_od > lim)
        TAG_FAIL(TAG_ESHAPE, "node or entry counts exceed the int32 index range");
    if ((s->e_oo && (!d->oo_src || !d->oo_dst)) || (s->e_dd && (!d->dd_a || !d->dd_b)) ||
        (s->e_od && (!d->od_op || !d->od_dev)))
        TAG_FAIL(TAG_EINVAL, "edge arrays must be non-NULL when their counts are positive");
    s->rows[0] = s->rows[1] = s->n_op;
    s->rows[2] = s->rows[3] = s->n_dev;
    s->nnz[0] = 2 * s->e_oo;
    s->nnz[1] = s->nnz[2] = s->e_od;
    s->nnz[3] = 2 * s->e_dd;
    return TAG_OK;
}

int64_t count_tiles(const tag_graph_desc *d) {
    int64_t n = 0;
    for (int32_t g = 0; g < d->n_graphs; ++g) n += (d->n_op[g] + kOpTile - 1) / kOpTile;
    return n;
}

int64_t count_groups(const tag_graph_desc *d) {
    int64_t n = 0;
    for (int32_t g = 0; g < d->n_graphs; ++g) {
        const int64_t nt = (d->n_op[g] + kOpTile - 1) / kOpTile;
        const int32_t tpg = tiles_per_group(nt);
        n += (nt + tpg - 1) / tpg;
    }
    return n;
}

// persistent metadata block inside the CSR buffer (one host->device copy):
// op_off [G+1] | dev_off [G+1] | tile_off [G+1] | group_off [G+1] |
// tiles [n_tiles][3] | groups [n_groups][2]
struct CsrLayout {
    int32_t *rowptr[4], *col[4], *eid[4];
    int32_t *oo_head;
    int32_t *meta;
    int32_t *op_off, *dev_off, *tile_off, *group_off, *tiles, *groups;
    size_t meta_ints;
};
// scratch: counters of all buckets, then the flags (one clear); link offsets (one copy)
struct TmpLayout {
    int32_t *cnt_all;          // [sum(rows + 1)] then flags [FLAG_COUNT]
    int64_t cnt_ints;
    int32_t *cnt[4], *flags;
    int32_t *tcol[4], *teid[4], *rowof[4];
    int32_t *tile_sums;
    int64_t *links;            // oo_off [G+1] | dd_off [G+1] | od_off [G+1]
};

size_t carve_csr(const Sizes &s, int64_t n_tiles, int64_t n_groups, void *base, CsrLayout *L) {
    Carver c(base);
    for (int b = 0; b < 4; ++b) {
        L->rowptr[b] = c.take<int32_t>(s.rows[b] + 1);
        L->col[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        L->eid[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
    }
    L->oo_head = c.take<int32_t>(std::max<int64_t>(s.e_oo, 1));
    const size_t nt = (size_t)std::max<int64_t>(n_tiles, 1);
    L->meta_ints = 4 * (size_t)(s.G + 1) + 3 * nt + 2 * (size_t)std::max<int64_t>(n_groups, 1);
    L->meta = c.take<int32_t>(L->meta_ints);
    L->op_off = L->meta ? L->meta : nullptr;
    L->dev_off = L->meta ? L->meta + (s.G + 1) : nullptr;
    L->tile_off = L->meta ? L->meta + 2 * (s.G + 1) : nullptr;
    L->group_off = L->meta ? L->meta + 3 * (s.G + 1) : nullptr;
    L->tiles = L->meta ? L->meta + 4 * (s.G + 1) : nullptr;
    L->groups = L->meta ? L->meta + 4 * (s.G + 1) + 3 * nt : nullptr;
    return c.used;
}

size_t carve_tmp(const Sizes &s, void *base, TmpLayout *L) {
    Carver c(base);
    L->cnt_ints = 0;
    for (int b = 0; b < 4; ++b) L->cnt_ints += s.rows[b] + 1;
    L->cnt_all = c.take<int32_t>(L->cnt_ints + FLAG_COUNT);
    int64_t off = 0;
    for (int b = 0; b < 4; ++b) {
        L->cnt[b] = L->cnt_all ? L->cnt_all + off : nullptr;
        off += s.rows[b] + 1;
    }
    L->flags = L->cnt_all ? L->cnt_all + L->cnt_ints : nullptr;
    int64_t max_tiles = 1;
    for (int b = 0; b < 4; ++b) {
        L->tcol[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        L->teid[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        L->rowof[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        max_tiles = std::max<int64_t>(max_tiles, (s.rows[b] + 1 + kScanTile - 1) / kScanTile);
    }
    L->tile_sums = c.take<int32_t>(max_tiles + 1);
    L->links = c.take<int64_t>(3 * (size_t)(s.G + 1));
    return c.used;
}

// exclusive scan of cnt[0..n) into rp[0..n], rp[n] = total (large arrays)
void enqueue_scan(const int32_t *cnt, int64_t n, int32_t *rp, int32_t *tile_sums, hipStream_t st) {
    int64_t m = n + 1;   // scan n+1 values (cnt[n] is 0) so rp[n] = total
    unsigned tiles = (unsigned)((m + kScanTile - 1) / kScanTile);
    scan_tiles<<<tiles, kThreads, 0, st>>>(cnt, m, rp, tile_sums);
    scan_sums<<<1, kThreads, 0, st>>>(tile_sums, tiles, tile_sums + tiles);
    scan_add<<<grid_for(m, INT32_MAX), kThreads, 0, st>>>(rp, m, tile_sums);
}

}  // namespace
}  // namespace tag

using namespace tag;

extern "C" const char *tag_last_error(void) { return tag::g_last_error.c_str(); }
extern "C" const char *tag_version(void) { return "tag-mi355x 0.1 (gfx950)"; }

extern "C" tag_status tag_graph_plan(const tag_graph_desc *desc, size_t *csr_bytes, size_t *tmp_bytes) {
    clear_error();
    if (!csr_bytes || !tmp_bytes) TAG_FAIL(TAG_EINVAL, "output size pointers must be non-NULL");
    Sizes s;
    tag_status st = check_desc(desc, &s);
    if (st != TAG_OK) return st;
    CsrLayout cl;
    TmpLayout tl;
    *csr_bytes = carve_csr(s, count_tiles(desc), count_groups(desc), nullptr, &cl);
    *tmp_bytes = carve_tmp(s, nullptr, &tl);
    return TAG_OK;
}

extern "C" tag_status tag_graph_build(const tag_graph_desc *desc, void *csr_buf, size_t csr_bytes,
                                      void *tmp_buf, size_t tmp_bytes, void *hip_stream,
                                      tag_graph **out) {
    clear_error();
    if (!out) TAG_FAIL(TAG_EINVAL, "out must be non-NULL");
    *out = nullptr;
    Sizes s;
    tag_status st = check_desc(desc, &s);
    if (st != TAG_OK) return st;
    if (!csr_buf || !tmp_buf) TAG_FAIL(TAG_EINVAL, "csr_buf and tmp_buf must be non-NULL");
    CsrLayout cl;
    TmpLayout tl;
    const int64_t n_tiles = count_tiles(desc), n_groups = count_groups(desc);
    if (carve_csr(s, n_tiles, n_groups, nullptr, &cl) > csr_bytes)
        TAG_FAIL(TAG_ENOSPACE, "csr buffer too small (see tag_graph_plan)");
    if (carve_tmp(s, nullptr, &tl) > tmp_bytes) TAG_FAIL(TAG_ENOSPACE, "tmp buffer too small (see tag_graph_plan)");
    carve_csr(s, n_tiles, n_groups, csr_buf, &cl);
    carve_tmp(s, tmp_buf, &tl);
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);

    auto *g = new tag_graph();
    g->G = s.G;
    g->max_dev = s.max_dev;
    g->n_op = s.n_op; g->n_dev = s.n_dev;
    g->e_oo = s.e_oo; g->e_dd = s.e_dd; g->e_od = s.e_od;
    g->op_off.assign(s.G + 1, 0);
    g->dev_off.assign(s.G + 1, 0);
    for (int32_t i = 0; i < s.G; ++i) {
        g->op_off[i + 1] = g->op_off[i] + desc->n_op[i];
        g->dev_off[i + 1] = g->dev_off[i] + desc->n_dev[i];
    }
    for (int b = 0; b < 4; ++b) { g->rows[b] = s.rows[b]; g->nnz[b] = s.nnz[b]; }
    if (hipGetDevice(&g->device) != hipSuccess) g->device = 0;

    // host staging of the persistent metadata and of the link offsets
    std::vector<int32_t> meta(cl.meta_ints, 0);
    std::vector<int64_t> links(3 * (size_t)(s.G + 1));
    {
        int32_t *op_off = meta.data(), *dev_off = op_off + (s.G + 1), *tile_off = dev_off + (s.G + 1);
        int32_t *group_off = tile_off + (s.G + 1);
        int32_t *tiles = group_off + (s.G + 1);
        int32_t *groups = tiles + 3 * std::max<int64_t>(n_tiles, 1);
        int32_t nt = 0, ng = 0;
        for (int32_t gi = 0; gi <= s.G; ++gi) {
            op_off[gi] = (int32_t)g->op_off[gi];
            dev_off[gi] = (int32_t)g->dev_off[gi];
        }
        for (int32_t gi = 0; gi < s.G; ++gi) {   // op tiles never cross a topology boundary
            tile_off[gi] = nt;
            int32_t cnt = 0;
            for (int32_t u = 0; u < desc->n_op[gi]; u += kOpTile, ++cnt, ++nt) {
                tiles[3 * nt] = op_off[gi] + u;
                tiles[3 * nt + 1] = std::min<int32_t>(kOpTile, desc->n_op[gi] - u);
                tiles[3 * nt + 2] = gi;
            }
            g->max_tiles = std::max(g->max_tiles, cnt);
            group_off[gi] = ng;
            const int32_t tpg = tiles_per_group(cnt);
            int32_t gcnt = 0;
            for (int32_t k = 0; k < cnt; k += tpg, ++gcnt, ++ng) {
                groups[2 * ng] = tile_off[gi] + k;
                groups[2 * ng + 1] = std::min(tpg, cnt - k);
            }
            g->max_groups = std::max(g->max_groups, gcnt);
        }
        tile_off[s.G] = nt;
        group_off[s.G] = ng;
        g->n_tiles = nt;
        g->n_groups = ng;
        for (int32_t gi = 0; gi <= s.G; ++gi) {
            links[gi] = desc->oo_off[gi];
            links[(s.G + 1) + gi] = desc->dd_off[gi];
            links[2 * (s.G + 1) + gi] = desc->od_off[gi];
        }
    }

    auto fail = [&](tag_status code, const std::string &msg) {
        delete g;
        set_error(msg);
        return code;
    };
#define BUILD_HIP(expr)                                                                       \
    do {                                                                                      \
        hipError_t e_ = (expr);                                                               \
        if (e_ != hipSuccess) return fail(TAG_EHIP, std::string(#expr ": ") + hipGetErrorString(e_)); \
    } while (0)

    BUILD_HIP(hipMemcpyAsync(cl.meta, meta.data(), sizeof(int32_t) * meta.size(), hipMemcpyHostToDevice, stream));
    BUILD_HIP(hipMemcpyAsync(tl.links, links.data(), sizeof(int64_t) * links.size(), hipMemcpyHostToDevice, stream));

    Buckets B{};
    for (int b = 0; b < 4; ++b) {
        B.rows[b] = s.rows[b]; B.nnz[b] = s.nnz[b];
        B.cnt[b] = tl.cnt[b]; B.rp[b] = cl.rowptr[b];
        B.tcol[b] = tl.tcol[b]; B.teid[b] = tl.teid[b]; B.rowof[b] = tl.rowof[b];
        B.col[b] = cl.col[b]; B.eid[b] = cl.eid[b];
    }
    const int32_t priv = s.n_dev <= kPrivRows ? 1 : 0;
    EdgeArgs ea{};
    ea.G = s.G;
    ea.n_dev = (int32_t)std::min<int64_t>(s.n_dev, kPrivRows);
    ea.B = B;
    ea.flags = tl.flags;
    ea.oo_head = cl.oo_head;
    const int64_t *oo_off = tl.links, *dd_off = tl.links + (s.G + 1), *od_off = tl.links + 2 * (s.G + 1);
    // op->op: (row = consumer, col = producer) and the reverse, both into B0
    ea.rel[0] = Rel{desc->oo_src, desc->oo_dst, oo_off, cl.op_off, cl.op_off, s.e_oo, 1, 0, 0, 0, 0};
    // dev-dev: both directions into B3 (device rows)
    ea.rel[1] = Rel{desc->dd_a, desc->dd_b, dd_off, cl.dev_off, cl.dev_off, s.e_dd, 1, 3, 3, priv, priv};
    // op-dev (op a, dev b): B2 row = dev (device rows), B1 row = op
    ea.rel[2] = Rel{desc->od_op, desc->od_dev, od_off, cl.op_off, cl.dev_off, s.e_od, 0, 2, 1, priv, 0};
    ea.blk_off[0] = 0;
    ea.blk_off[1] = (s.e_oo + kThreads - 1) / kThreads;
    ea.blk_off[2] = ea.blk_off[1] + (s.e_dd + kThreads - 1) / kThreads;
    ea.blk_off[3] = ea.blk_off[2] + (s.e_od + kThreads - 1) / kThreads;
    const int64_t nnz_all = s.nnz[0] + s.nnz[1] + s.nnz[2] + s.nnz[3];

    prof_begin(TAG_STAGE_GRAPH_BUILD, stream);
    fill_i32<<<grid_for(tl.cnt_ints + FLAG_COUNT), kThreads, 0, stream>>>(tl.cnt_all, tl.cnt_ints + FLAG_COUNT, 0);
    if (ea.blk_off[3] > 0) edges_pass<0><<<(unsigned)ea.blk_off[3], kThreads, 0, stream>>>(ea);
    if (std::max(s.rows[0], s.rows[2]) + 1 <= kSmallScan) {
        scan_buckets<<<4, kThreads, 0, stream>>>(B);   // also zeroes the counters
    } else {
        for (int b = 0; b < 4; ++b) enqueue_scan(tl.cnt[b], s.rows[b], cl.rowptr[b], tl.tile_sums, stream);
        fill_i32<<<grid_for(tl.cnt_ints), kThreads, 0, stream>>>(tl.cnt_all, tl.cnt_ints, 0);
    }
    if (ea.blk_off[3] > 0) edges_pass<1><<<(unsigned)ea.blk_off[3], kThreads, 0, stream>>>(ea);
    if (nnz_all > 0) {
        const int64_t r1 = s.rows[0], r2 = r1 + s.rows[1], r3 = r2 + s.rows[2], rtot = r3 + s.rows[3];
        const int64_t n_short = (rtot + kThreads / 64 - 1) / (kThreads / 64);
        // op<-op and dev<-op rows can be long; valid op<-dev and dev<-dev rows have at most 64 entries
        const int64_t n_long = s.nnz[0] + s.nnz[2] > 0 ? s.rows[0] + s.rows[2] : 0;
        // bitmap sized for the largest topology (sources of both buckets are ops)
        int32_t rmax = 1;
        for (int32_t gi = 0; gi < s.G; ++gi) rmax = std::max(rmax, desc->n_op[gi]);
        rmax = std::min(rmax, kBitmapRange);
        const size_t lds = sizeof(int32_t) * (2 * (size_t)((rmax + 31) / 32) + (size_t)rmax);
        rank_all<<<(unsigned)(n_short + n_long), kThreads, lds, stream>>>(B, r1, r2, r3, rtot, n_short, cl.op_off,
                                                                           cl.dev_off, s.G, rmax, tl.flags);
    }
    prof_end(TAG_STAGE_GRAPH_BUILD, stream);
    {
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return fail(TAG_EHIP, std::string("graph build launch: ") + hipGetErrorString(e));
    }
    int32_t flags[FLAG_COUNT];
    BUILD_HIP(hipMemcpyAsync(flags, tl.flags, sizeof(flags), hipMemcpyDeviceToHost, stream));
    BUILD_HIP(hipStreamSynchronize(stream));
    if (flags[FLAG_RANGE]) return fail(TAG_ERANGE, "a node id is out of range for its topology");
    if (flags[FLAG_DUP]) return fail(TAG_EDUP, "self link, duplicate pair, or a tensor link given in both directions");
    for (int b = 0; b < 4; ++b) {
        g->rowptr[b] = cl.rowptr[b];
        g->col[b] = cl.col[b];
        g->eid[b] = cl.eid[b];
        g->max_degree[b] = flags[FLAG_MAXDEG + b];
    }
    g->oo_head = cl.oo_head;
    g->op_off_d = cl.op_off;
    g->dev_off_d = cl.dev_off;
    g->tiles_d = cl.tiles;
    g->tile_off_d = cl.tile_off;
    g->groups_d = cl.groups;
    g->group_off_d = cl.group_off;
    *out = g;
#undef BUILD_HIP
    return TAG_OK;
}

extern "C" tag_status tag_graph_get_info(const tag_graph *g, tag_graph_info *info) {
    clear_error();
    if (!g || !info) TAG_FAIL(TAG_EINVAL, "graph and info must be non-NULL");
    info->n_graphs = g->G;
    info->max_dev = g->max_dev;
    info->n_op = g->n_op; info->n_dev = g->n_dev;
    info->e_oo = g->e_oo; info->e_dd = g->e_dd; info->e_od = g->e_od;
    for (int b = 0; b < 4; ++b) {
        info->rows[b] = g->rows[b];
        info->nnz[b] = g->nnz[b];
        info->max_degree[b] = g->max_degree[b];
    }
    return TAG_OK;
}

extern "C" tag_status tag_graph_export(const tag_graph *g, int32_t bucket, int32_t *rowptr_host,
                                       int32_t *col_host, int32_t *eid_host) {
    clear_error();
    if (!g) TAG_FAIL(TAG_EINVAL, "graph is NULL");
    if (bucket < 0 || bucket > 3) TAG_FAIL(TAG_EINVAL, "bucket must be 0..3");
    if (rowptr_host)
        TAG_HIP_CHECK(hipMemcpy(rowptr_host, g->rowptr[bucket], sizeof(int32_t) * (g->rows[bucket] + 1),
                                hipMemcpyDeviceToHost));
    if (col_host && g->nnz[bucket])
        TAG_HIP_CHECK(hipMemcpy(col_host, g->col[bucket], sizeof(int32_t) * g->nnz[bucket], hipMemcpyDeviceToHost));
    if (eid_host && g->nnz[bucket])
        TAG_HIP_CHECK(hipMemcpy(eid_host, g->eid[bucket], sizeof(int32_t) * g->nnz[bucket], hipMemcpyDeviceToHost));
    return TAG_OK;
}

extern "C" void tag_graph_destroy(tag_graph *g) { delete g; }
