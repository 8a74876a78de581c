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
// Pipeline (all on the caller's stream): fill counters, count per-row
// degrees with integer atomics while validating ids, exclusive scan to row
// pointers, scatter with per-row atomic cursors (arbitrary order inside a
// row), then an exact per-row rank sort: each entry's final slot is the
// number of entries of its row with a smaller (source, edge) key.  The rank
// pass also detects repeated (row, source) pairs.  One stream sync at the
// end reads the validation flags and per-bucket maximum degrees.
#include <algorithm>
#include <mutex>

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

// flags layout in the tmp buffer
enum { FLAG_RANGE = 0, FLAG_DUP = 1, FLAG_MAXDEG = 4 /* 4 entries */, FLAG_COUNT = 8 };

__global__ void fill_i32(int32_t *p, int64_t n, int32_t v) {
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

// topology owning entry i of a prefix-offset array off[0..G]
__device__ __forceinline__ int32_t owner(const int64_t *off, int32_t G, int64_t i) {
    int32_t lo = 0, hi = G;   // find last g with off[g] <= i
    while (hi - lo > 1) {
        int32_t mid = (lo + hi) >> 1;
        if (off[mid] <= i) lo = mid; else hi = mid;
    }
    return lo;
}

struct EdgeArgs {
    const int32_t *a, *b;      // per-edge endpoints (local ids)
    const int64_t *off;        // device copy of the link prefix offsets [G+1]
    const int32_t *a_off;      // node prefix offsets of endpoint a's type [G+1]
    const int32_t *b_off;      // node prefix offsets of endpoint b's type [G+1]
    int64_t n_edges;
    int32_t G;
    int32_t same_type;         // 1: a and b are the same node type (self links rejected)
    // bucket fed as (row = b, col = a) and bucket fed as (row = a, col = b)
    int32_t *cnt_ba, *cnt_ab;
    const int32_t *rp_ba, *rp_ab;
    int32_t *col_ba, *eid_ba, *rowof_ba;
    int32_t *col_ab, *eid_ab, *rowof_ab;
};

// mode 0: count degrees; mode 1: scatter entries
template <int MODE>
__global__ void edges_pass(EdgeArgs A, int32_t *flags) {
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < A.n_edges; i += stride) {
        int32_t g = owner(A.off, A.G, i);
        int32_t la = A.a[i], lb = A.b[i];
        int32_t na = A.a_off[g + 1] - A.a_off[g], nb = A.b_off[g + 1] - A.b_off[g];
        if (la < 0 || la >= na || lb < 0 || lb >= nb) {
            if (MODE == 0) atomicOr(&flags[FLAG_RANGE], 1);
            continue;
        }
        if (A.same_type && la == lb) {
            if (MODE == 0) atomicOr(&flags[FLAG_DUP], 1);
            continue;
        }
        int32_t ga = A.a_off[g] + la, gb = A.b_off[g] + lb;
        if (MODE == 0) {
            atomicAdd(&A.cnt_ba[gb], 1);
            atomicAdd(&A.cnt_ab[ga], 1);
        } else {
            int32_t p = A.rp_ba[gb] + atomicAdd(&A.cnt_ba[gb], 1);
            A.col_ba[p] = ga; A.eid_ba[p] = (int32_t)i; A.rowof_ba[p] = gb;
            int32_t q = A.rp_ab[ga] + atomicAdd(&A.cnt_ab[ga], 1);
            A.col_ab[q] = gb; A.eid_ab[q] = (int32_t)i; A.rowof_ab[q] = ga;
        }
    }
}

// ---- exclusive scan of int32 counts (n + 1 outputs, out[n] = total) ----
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, int32_t *total, int32_t *sh) {
    // sh: kThreads ints
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

// ---- exact per-row rank sort ----
constexpr int kShortRow = 256;        // rows up to this length: per-entry rank
constexpr int kBitmapRange = 16384;   // source-id range sorted through an LDS bitmap

// Only the first rp[n_rows] slots hold entries: links rejected during the
// count pass (bad ids, self links) were never scattered.  Rows longer than
// kShortRow are left to rank_long_rows.
__global__ void rank_rows(const int32_t *rp, int64_t n_rows, const int32_t *tcol, const int32_t *teid,
                          const int32_t *rowof, int64_t nnz, int32_t *col, int32_t *eid,
                          int32_t *flags, int bucket) {
    int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (p >= nnz || p >= rp[n_rows]) return;
    int32_t r = rowof[p];
    int32_t beg = rp[r], end = rp[r + 1];
    if (end - beg > kShortRow) return;
    int32_t c = tcol[p], e = teid[p];
    int32_t rank = 0, dup = 0;
    for (int32_t q = beg; q < end; ++q) {
        int32_t cq = tcol[q], eq = teid[q];
        rank += (cq < c) || (cq == c && eq < e);
        dup |= (cq == c) && (q != p);
    }
    col[beg + rank] = c;
    eid[beg + rank] = e;
    if (dup) atomicOr(&flags[FLAG_DUP], 1);
    if (rank == 0) atomicMax(&flags[FLAG_MAXDEG + bucket], end - beg);
}

// One block per long row.  Sources of a row all belong to the row's
// topology, so a bitmap over that topology's source-id range sorts the row
// by source id (sources are unique in a valid row; a repeated source is
// caught by the atomic OR).  Ranges beyond kBitmapRange fall back to the
// per-entry rank inside the block.
__global__ void __launch_bounds__(256) rank_long_rows(const int32_t *rp, const int32_t *tcol, const int32_t *teid,
                                                      int32_t *col, int32_t *eid, int32_t *flags, int bucket,
                                                      const int32_t *row_off, const int32_t *src_off, int32_t G) {
    __shared__ uint32_t bm[kBitmapRange / 32];
    __shared__ int32_t wpre[kBitmapRange / 32];
    __shared__ int32_t eid_of[kBitmapRange];
    __shared__ int32_t scan[256];
    const int32_t r = blockIdx.x;
    const int32_t beg = rp[r], end = rp[r + 1];
    if (end - beg <= kShortRow) return;
    int32_t lo = 0, hi = G;
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (row_off[mid] <= r) lo = mid; else hi = mid;
    }
    const int32_t base = src_off[lo], range = src_off[lo + 1] - base;
    if (threadIdx.x == 0) atomicMax(&flags[FLAG_MAXDEG + bucket], end - beg);
    if (range > kBitmapRange) {
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
        uint32_t b = bm[w];
        int32_t pos = beg + wpre[w];
        while (b) {
            const int k = __ffs(b) - 1;
            b &= b - 1u;
            const int32_t c = w * 32 + k;
            col[pos] = base + c;
            eid[pos] = eid_of[c];
            ++pos;
        }
    }
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

struct CsrLayout {
    int32_t *rowptr[4], *col[4], *eid[4];
    int32_t *op_off, *dev_off;
    int32_t *tiles, *tile_off;
};

int64_t count_tiles(const tag_graph_desc *d) {
    int64_t n = 0;
    for (int32_t g = 0; g < d->n_graphs; ++g) n += (d->n_op[g] + kOpTile - 1) / kOpTile;
    return n;
}
struct TmpLayout {
    int32_t *cnt[4], *tcol[4], *teid[4], *rowof[4];
    int32_t *tile_sums;
    int32_t *flags;
    int64_t *oo_off, *dd_off, *od_off;
};

size_t carve_csr(const Sizes &s, int64_t n_tiles, void *base, CsrLayout *L) {
    Carver c(base);
    for (int b = 0; b < 4; ++b) {
        L->rowptr[b] = c.take<int32_t>(s.rows[b] + 1);
        L->col[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        L->eid[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
    }
    L->op_off = c.take<int32_t>(s.G + 1);
    L->dev_off = c.take<int32_t>(s.G + 1);
    L->tiles = c.take<int32_t>(3 * std::max<int64_t>(n_tiles, 1));
    L->tile_off = c.take<int32_t>(s.G + 1);
    return c.used;
}

size_t carve_tmp(const Sizes &s, void *base, TmpLayout *L) {
    Carver c(base);
    int64_t max_tiles = 1;
    for (int b = 0; b < 4; ++b) {
        L->cnt[b] = c.take<int32_t>(s.rows[b] + 1);
        L->tcol[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        L->teid[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        L->rowof[b] = c.take<int32_t>(std::max<int64_t>(s.nnz[b], 1));
        max_tiles = std::max<int64_t>(max_tiles, (s.rows[b] + 1 + kScanTile - 1) / kScanTile);
    }
    L->tile_sums = c.take<int32_t>(max_tiles + 1);
    L->flags = c.take<int32_t>(FLAG_COUNT);
    L->oo_off = c.take<int64_t>(s.G + 1);
    L->dd_off = c.take<int64_t>(s.G + 1);
    L->od_off = c.take<int64_t>(s.G + 1);
    return c.used;
}

// exclusive scan of cnt[0..n) into rp[0..n], rp[n] = total
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
    *csr_bytes = carve_csr(s, count_tiles(desc), nullptr, &cl);
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
    const int64_t n_tiles = count_tiles(desc);
    if (carve_csr(s, n_tiles, nullptr, &cl) > csr_bytes) TAG_FAIL(TAG_ENOSPACE, "csr buffer too small (see tag_graph_plan)");
    if (carve_tmp(s, nullptr, &tl) > tmp_bytes) TAG_FAIL(TAG_ENOSPACE, "tmp buffer too small (see tag_graph_plan)");
    carve_csr(s, n_tiles, csr_buf, &cl);
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
    std::vector<int32_t> op_off32(g->op_off.begin(), g->op_off.end());
    std::vector<int32_t> dev_off32(g->dev_off.begin(), g->dev_off.end());
    // op tiles never cross a topology boundary
    std::vector<int32_t> tiles;
    std::vector<int32_t> tile_off(s.G + 1, 0);
    tiles.reserve(3 * n_tiles);
    for (int32_t gi = 0; gi < s.G; ++gi) {
        int32_t nt = 0;
        for (int32_t u = 0; u < desc->n_op[gi]; u += kOpTile, ++nt) {
            tiles.push_back(static_cast<int32_t>(g->op_off[gi]) + u);
            tiles.push_back(std::min<int32_t>(kOpTile, desc->n_op[gi] - u));
            tiles.push_back(gi);
        }
        tile_off[gi + 1] = tile_off[gi] + nt;
        g->max_tiles = std::max(g->max_tiles, nt);
    }
    g->n_tiles = static_cast<int32_t>(n_tiles);
    for (int b = 0; b < 4; ++b) { g->rows[b] = s.rows[b]; g->nnz[b] = s.nnz[b]; }
    if (hipGetDevice(&g->device) != hipSuccess) g->device = 0;

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

    BUILD_HIP(hipMemcpyAsync(cl.op_off, op_off32.data(), sizeof(int32_t) * (s.G + 1), hipMemcpyHostToDevice, stream));
    BUILD_HIP(hipMemcpyAsync(cl.dev_off, dev_off32.data(), sizeof(int32_t) * (s.G + 1), hipMemcpyHostToDevice, stream));
    BUILD_HIP(hipMemcpyAsync(cl.tiles, tiles.data(), sizeof(int32_t) * tiles.size(), hipMemcpyHostToDevice, stream));
    BUILD_HIP(hipMemcpyAsync(cl.tile_off, tile_off.data(), sizeof(int32_t) * (s.G + 1), hipMemcpyHostToDevice, stream));
    BUILD_HIP(hipMemcpyAsync(tl.oo_off, desc->oo_off, sizeof(int64_t) * (s.G + 1), hipMemcpyHostToDevice, stream));
    BUILD_HIP(hipMemcpyAsync(tl.dd_off, desc->dd_off, sizeof(int64_t) * (s.G + 1), hipMemcpyHostToDevice, stream));
    BUILD_HIP(hipMemcpyAsync(tl.od_off, desc->od_off, sizeof(int64_t) * (s.G + 1), hipMemcpyHostToDevice, stream));

    prof_begin(TAG_STAGE_GRAPH_BUILD, stream);
    for (int b = 0; b < 4; ++b)
        fill_i32<<<grid_for(s.rows[b] + 1), kThreads, 0, stream>>>(tl.cnt[b], s.rows[b] + 1, 0);
    fill_i32<<<1, kThreads, 0, stream>>>(tl.flags, FLAG_COUNT, 0);

    // op->op: row = consumer / col = producer (B0), and the reverse (B0)
    EdgeArgs eo{desc->oo_src, desc->oo_dst, tl.oo_off, cl.op_off, cl.op_off, s.e_oo, s.G, 1,
                tl.cnt[0], tl.cnt[0], cl.rowptr[0], cl.rowptr[0],
                tl.tcol[0], tl.teid[0], tl.rowof[0], tl.tcol[0], tl.teid[0], tl.rowof[0]};
    // op-dev: (op a, dev b): B2 row = dev, col = op; B1 row = op, col = dev
    EdgeArgs ep{desc->od_op, desc->od_dev, tl.od_off, cl.op_off, cl.dev_off, s.e_od, s.G, 0,
                tl.cnt[2], tl.cnt[1], cl.rowptr[2], cl.rowptr[1],
                tl.tcol[2], tl.teid[2], tl.rowof[2], tl.tcol[1], tl.teid[1], tl.rowof[1]};
    // dev-dev: both directions into B3
    EdgeArgs ed{desc->dd_a, desc->dd_b, tl.dd_off, cl.dev_off, cl.dev_off, s.e_dd, s.G, 1,
                tl.cnt[3], tl.cnt[3], cl.rowptr[3], cl.rowptr[3],
                tl.tcol[3], tl.teid[3], tl.rowof[3], tl.tcol[3], tl.teid[3], tl.rowof[3]};
    EdgeArgs *passes[3] = {&eo, &ep, &ed};
    for (EdgeArgs *a : passes)
        if (a->n_edges) edges_pass<0><<<grid_for(a->n_edges), kThreads, 0, stream>>>(*a, tl.flags);
    for (int b = 0; b < 4; ++b) {
        enqueue_scan(tl.cnt[b], s.rows[b], cl.rowptr[b], tl.tile_sums, stream);
        fill_i32<<<grid_for(s.rows[b] + 1), kThreads, 0, stream>>>(tl.cnt[b], s.rows[b] + 1, 0);
    }
    for (EdgeArgs *a : passes)
        if (a->n_edges) edges_pass<1><<<grid_for(a->n_edges), kThreads, 0, stream>>>(*a, tl.flags);
    for (int b = 0; b < 4; ++b)
        if (s.nnz[b])
            rank_rows<<<(unsigned)((s.nnz[b] + kThreads - 1) / kThreads), kThreads, 0, stream>>>(
                cl.rowptr[b], s.rows[b], tl.tcol[b], tl.teid[b], tl.rowof[b], s.nnz[b], cl.col[b], cl.eid[b],
                tl.flags, b);
    // op<-op and dev<-op rows can be long; op<-dev and dev<-dev rows have at most 64 entries
    if (s.nnz[0])
        rank_long_rows<<<(unsigned)s.rows[0], kThreads, 0, stream>>>(cl.rowptr[0], tl.tcol[0], tl.teid[0], cl.col[0],
                                                                      cl.eid[0], tl.flags, 0, cl.op_off, cl.op_off, s.G);
    if (s.nnz[2])
        rank_long_rows<<<(unsigned)s.rows[2], kThreads, 0, stream>>>(cl.rowptr[2], tl.tcol[2], tl.teid[2], cl.col[2],
                                                                      cl.eid[2], tl.flags, 2, cl.dev_off, cl.op_off, s.G);
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
    g->op_off_d = cl.op_off;
    g->dev_off_d = cl.dev_off;
    g->tiles_d = cl.tiles;
    g->tile_off_d = cl.tile_off;
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
