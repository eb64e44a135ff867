// Balanced k-means of neuron feature rows: MoEfication's clustering step
// (Sec. 2.2), which groups the d_ff intermediate neurons into E experts of
// exactly d_ff / E neurons and so defines the permutation Pi of
// Eq. (permuted_weights).  Lloyd's iteration under the balance constraint
// (the constrained k-means the paper cites):
//
//   assignment  minimise sum_i ||x_i - mu_a(i)||^2 with every cluster holding
//               exactly m = n / k rows: a transportation problem, solved
//               exactly by an ascending-price auction on the k cluster prices
//               lambda (dual variables).  Each round every row takes its exact
//               argmax of -s_ij - lambda_j (s_ij = ||mu_j||^2 - 2 x_i . mu_j,
//               the row's own ||x_i||^2 does not change the choice); every
//               over-full cluster raises its price by the (m+1)-th largest
//               margin (best minus second-best value) of its rows plus eps.
//               When no cluster is over-full all hold exactly m rows, and an
//               argmax assignment that is balanced is optimal by LP duality,
//               whatever eps was; eps only ends price wars, so it decays
//               geometrically (0.3 scale * 0.9^r, floor 2^-22 scale).  Small
//               steps cannot move a price far, so after kKmAuctionRounds
//               rounds the rest of the excess is routed by successive
//               shortest paths on the k-node cluster graph (edge a -> b: the
//               cheapest move of one of a's rows to b, minus the price
//               difference, >= 0 since every row sits at its argmax); each
//               augmentation moves one unit from an over-full to an
//               under-full cluster and updates the prices by the Dijkstra
//               distances (Johnson potentials), which keeps every row at its
//               argmax -- so the result stays exactly optimal.
//   update      mu_j = mean of the rows of cluster j (ascending row order).
//   Pi          clusters in index order, rows ascending inside each.
//
// Kernels: km_xnorm_k (||x_i||^2, fp64), km_split_k (mu as three bf16 parts
// mu = h + m + l exactly, and ||mu_j||^2), km_dist_k (s = ||mu||^2 - 2 F mu^T
// with bf16 MFMA 16x16x32 on the exact bf16 features and the three parts:
// products exact, fp32 accumulation, HBM-bound on F), km_bid_k / km_price_k
// (one auction round each), km_ssp_k (the shortest-path finish, one
// workgroup), km_objective_k, km_perm_k, km_update_k.
#include <utility>

#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kKmMaxK = 256;
constexpr int kKmMaxN = 65536;
constexpr int kKmMaxD = 16384;
constexpr int kKmCols = 64;            // columns of mu staged in LDS per chunk
constexpr int kKmDistWaves = 8;        // km_dist_k: 8 wavefronts x 16 rows
constexpr int kKmBidThreads = 256;
constexpr int kKmPriceThreads = 256;
constexpr int kKmAuctionRounds = 128;  // price rounds before the shortest-path finish
constexpr int kKmBatch = 64;           // rounds enqueued between convergence checks
constexpr int kKmSspThreads = 1024;

struct KmWork {
    float *S;            // [k][n] s_ij
    double *xnorm;       // [n]
    float *list;         // [k][n] margins (rounded up to fp32) of each cluster's rows
    int32_t *memb;       // [k][n] the rows themselves (same order as list)
    double *lam;         // [k] cluster prices
    double *part;        // [bid workgroups] spread sums, then [bid workgroups] = the eps scale
    float *cn;           // [k] ||mu_j||^2
    uint16_t *mu3;       // [3][k][D] bf16 parts of mu
    int32_t *count;      // [k] rows whose argmax is j (this round)
    double *base;        // [k][k] shortest-path finish: min over a's rows of s_ib - s_ia
    int32_t *bidx;       // [k][k] the row attaining it (lowest index on ties)
    int32_t *pos;        // [n] a row's place in its cluster's member list
    int32_t *flags;      // [0..1] over-full clusters of round r (by parity), [2] done,
                         // [3] rounds the step took
};

inline int bid_blocks(int n) { return (n + kKmBidThreads / 4 - 1) / (kKmBidThreads / 4); }

size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

// Workspace carving (every region 256-byte aligned).
size_t km_layout(int n, int D, int k, KmWork *w, char *base) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *p = base ? base + off : nullptr;
        off += align_up(bytes);
        return p;
    };
    KmWork t;
    t.S = reinterpret_cast<float *>(take(sizeof(float) * (size_t)k * n));
    t.xnorm = reinterpret_cast<double *>(take(sizeof(double) * n));
    t.list = reinterpret_cast<float *>(take(sizeof(float) * (size_t)k * n));
    t.memb = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (size_t)k * n));
    t.lam = reinterpret_cast<double *>(take(sizeof(double) * k));
    t.part = reinterpret_cast<double *>(take(sizeof(double) * (bid_blocks(n) + 1)));
    t.cn = reinterpret_cast<float *>(take(sizeof(float) * k));
    t.mu3 = reinterpret_cast<uint16_t *>(take(sizeof(uint16_t) * 3 * (size_t)k * D));
    t.count = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * k));
    t.base = reinterpret_cast<double *>(take(sizeof(double) * (size_t)k * k));
    t.bidx = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (size_t)k * k));
    t.pos = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * n));
    t.flags = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * 4));
    if (w) *w = t;
    return off;
}

// ||x_i||^2 in fp64, one wavefront per row, lanes over 8-column groups in
// order, then a fixed butterfly.
__global__ __launch_bounds__(256) void km_xnorm_k(const uint16_t *__restrict__ F, int n, int D,
                                                  double *__restrict__ xnorm) {
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= n) return;
    const uint16_t *row = F + (size_t)i * D;
    double acc = 0.0;
    for (int c = 8 * lane; c < D; c += 512) {
        const uint4 v = ldg16(row + c);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const double a = bf16_to_f32((uint16_t)(w[q] & 0xFFFFu));
            const double b = bf16_to_f32((uint16_t)(w[q] >> 16));
            acc += a * a + b * b;
        }
    }
#pragma unroll
    for (int st = 32; st >= 1; st >>= 1) acc += __shfl_xor(acc, st, 64);
    if (lane == 0) xnorm[i] = acc;
}

// mu_j as three bf16 parts (h = bf16(mu), m = bf16(mu - h), l = bf16(mu - h - m),
// each difference exact in fp32) and ||mu_j||^2 (fp64 in a fixed order,
// stored fp32).  One workgroup per centroid.
__global__ __launch_bounds__(256) void km_split_k(const float *__restrict__ mu, int k, int D,
                                                  uint16_t *__restrict__ mu3,
                                                  float *__restrict__ cn) {
    __shared__ double red[256];
    const int j = blockIdx.x, tid = threadIdx.x;
    double acc = 0.0;
    for (int c = tid; c < D; c += 256) {
        const float v = mu[(size_t)j * D + c];
        const uint16_t h = f32_to_bf16(v);
        const float r1 = v - bf16_to_f32(h);
        const uint16_t m = f32_to_bf16(r1);
        const uint16_t l = f32_to_bf16(r1 - bf16_to_f32(m));
        const size_t o = (size_t)j * D + c;
        mu3[o] = h;
        mu3[(size_t)k * D + o] = m;
        mu3[2 * (size_t)k * D + o] = l;
        acc += (double)v * v;
    }
    red[tid] = acc;
    __syncthreads();
    for (int s = 128; s >= 1; s >>= 1) {
        if (tid < s) red[tid] += red[tid + s];
        __syncthreads();
    }
    if (tid == 0) cn[j] = (float)red[0];
}

// s[j][i] = ||mu_j||^2 - 2 x_i . mu_j.  A workgroup owns 128 rows (16 per
// wavefront, the MFMA A operand straight from HBM, prefetched one chunk
// ahead); the three bf16 parts of mu, kKmCols columns at a time, are staged
// in LDS in B-operand order and shared by the 8 wavefronts.  NT = ceil(k/16)
// cluster tiles per wavefront.
template <int NT>
__global__ __launch_bounds__(64 * kKmDistWaves) void km_dist_k(const uint16_t *__restrict__ F,
                                                              int n, int D, int k,
                                                              const uint16_t *__restrict__ mu3,
                                                              const float *__restrict__ cn,
                                                              float *__restrict__ S) {
    // bs[part][tile][K-step of 32][lane]: 16 bytes per lane
    __shared__ uint4 bs[3][NT][kKmCols / 32][64];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int p = lane & 15, g = lane >> 4;
    const int i0 = blockIdx.x * (16 * kKmDistWaves) + wv * 16;
    const int row = min(i0 + p, n - 1);
    const uint16_t *frow = F + (size_t)row * D + 8 * g;
    f32x4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    constexpr int kSteps = kKmCols / 32;
    uint4 a[kSteps], an[kSteps];
#pragma unroll
    for (int s = 0; s < kSteps; ++s) a[s] = ldg16(frow + 32 * s);
    const size_t plane = (size_t)k * D;
    for (int c0 = 0; c0 < D; c0 += kKmCols) {
        // stage mu parts for columns c0 .. c0 + kKmCols - 1
        for (int e = tid; e < 3 * NT * kSteps * 64; e += 64 * kKmDistWaves) {
            const int l = e & 63, s = (e >> 6) % kSteps, t = (e >> 6) / kSteps % NT,
                      part = (e >> 6) / kSteps / NT;
            const int j = t * 16 + (l & 15);
            uint4 v = make_uint4(0, 0, 0, 0);
            if (j < k) v = ldg16(mu3 + part * plane + (size_t)j * D + c0 + 32 * s + 8 * (l >> 4));
            bs[part][t][s][l] = v;
        }
        if (c0 + kKmCols < D) {
#pragma unroll
            for (int s = 0; s < kSteps; ++s) an[s] = ldg16(frow + c0 + kKmCols + 32 * s);
        }
        __syncthreads();
#pragma unroll
        for (int s = 0; s < kSteps; ++s)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int part = 0; part < 3; ++part)
                    acc[t] = mfma16(a[s], bs[part][t][s][lane], acc[t]);
        __syncthreads();
#pragma unroll
        for (int s = 0; s < kSteps; ++s) a[s] = an[s];
    }
    // lane holds rows i0 + 4 g + q (q < 4) of cluster t * 16 + p
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int j = t * 16 + p;
        if (j >= k) continue;
        const float c = cn[j];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = i0 + 4 * g + q;
            if (i < n) S[(size_t)j * n + i] = c - 2.0f * acc[t][q];
        }
    }
}

// Auction state for one assignment step: prices 0, counts 0, flags clear.
__global__ void km_auction_init_k(int k, double *lam, int32_t *count, int32_t *flags) {
    const int t = threadIdx.x;
    for (int j = t; j < k; j += blockDim.x) {
        lam[j] = 0.0;
        count[j] = 0;
    }
    if (t < 4) flags[t] = 0;
}

// (best, its cluster, second best) of part of a row's clusters; merging two
// parts gives the same result in any order: the better best wins (lower
// cluster on equal values), the second is the larger of the kept second and
// the other best.
struct Best2 {
    double w1, w2;
    int j1;
    float smin, smax;
};
__device__ __forceinline__ Best2 merge_best2(Best2 a, Best2 b) {
    if (b.w1 > a.w1 || (b.w1 == a.w1 && b.j1 < a.j1)) {
        const Best2 t = a;
        a = b;
        b = t;
    }
    a.w2 = fmax(a.w2, b.w1);
    a.smin = fminf(a.smin, b.smin);
    a.smax = fmaxf(a.smax, b.smax);
    return a;
}
__device__ __forceinline__ Best2 shfl_best2(const Best2 &v, int st) {
    Best2 o;
    o.w1 = __shfl_xor(v.w1, st, 64);
    o.w2 = __shfl_xor(v.w2, st, 64);
    o.j1 = __shfl_xor(v.j1, st, 64);
    o.smin = __shfl_xor(v.smin, st, 64);
    o.smax = __shfl_xor(v.smax, st, 64);
    return o;
}

// Round r, bids: every row's argmax j1 of w_ij = -s_ij - lambda_j (first
// index on ties) and its margin w1 - w2 (w2 the best over the other
// clusters), rounded up to fp32 and appended, with the row, to cluster j1's
// lists; counts per cluster.  kBidLanes adjacent lanes share a row, each
// taking every kBidLanes-th cluster with its loads 32 at a time in flight, and
// their partial results are merged.  Exits at once when the previous round
// left no cluster over-full (the assignment then stands).
constexpr int kBidLanes = 4;
constexpr int kBidRows = kKmBidThreads / kBidLanes;  // rows per workgroup

__global__ __launch_bounds__(kKmBidThreads) void km_bid_k(const float *__restrict__ S, int n, int k,
                                                          int r, KmWork W,
                                                          int32_t *__restrict__ assign) {
    constexpr int kBatch = 32;  // a lane's clusters in flight at once (k <= 128: all of them)
    __shared__ double lam[kKmMaxK];
    __shared__ int cnt[kKmMaxK];
    __shared__ int base[kKmMaxK];
    __shared__ double spread[kBidRows];
    const int tid = threadIdx.x;
    if (W.flags[2]) return;
    if (r > 0 && W.flags[(r - 1) & 1] == 0) {
        if (blockIdx.x == 0 && tid == 0) {
            W.flags[2] = 1;
            W.flags[3] = r;
        }
        return;
    }
    if (blockIdx.x == 0 && tid == 0) W.flags[r & 1] = 0;
    for (int j = tid; j < k; j += kKmBidThreads) {
        lam[j] = W.lam[j];
        cnt[j] = 0;
    }
    __syncthreads();
    const int q = tid % kBidLanes, row = tid / kBidLanes;
    const int i = blockIdx.x * kBidRows + row;
    const bool valid = i < n;
    const int ii = min(i, n - 1);
    Best2 v{-INFINITY, -INFINITY, 0x7FFFFFFF, INFINITY, -INFINITY};
    for (int j0 = q; j0 < k; j0 += kBatch * kBidLanes) {
        float sv[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            sv[u] = S[(size_t)min(j0 + u * kBidLanes, k - 1) * n + ii];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int j = j0 + u * kBidLanes;
            if (j < k) {
                const double w = -(double)sv[u] - lam[j];
                const bool b1 = w > v.w1;  // ascending j within a lane: first wins ties
                v.w2 = b1 ? v.w1 : fmax(v.w2, w);
                v.w1 = b1 ? w : v.w1;
                v.j1 = b1 ? j : v.j1;
                v.smin = fminf(v.smin, sv[u]);
                v.smax = fmaxf(v.smax, sv[u]);
            }
        }
    }
#pragma unroll
    for (int st = 1; st < kBidLanes; st <<= 1) v = merge_best2(v, shfl_best2(v, st));
    const bool lead = q == 0 && valid;
    int slot = 0;
    if (lead) slot = atomicAdd(&cnt[v.j1], 1);
    __syncthreads();
    for (int j = tid; j < k; j += kKmBidThreads) base[j] = cnt[j] ? atomicAdd(&W.count[j], cnt[j]) : 0;
    __syncthreads();
    if (lead) {
        const double mg = v.w1 - v.w2;  // +inf when k == 1
        const int at = base[v.j1] + slot;
        assign[i] = v.j1;
        W.list[(size_t)v.j1 * n + at] = isinf(mg) ? 3.0e38f : __double2float_ru(mg);
        W.memb[(size_t)v.j1 * n + at] = i;
        W.pos[i] = at;
    }
    if (r == 0) {  // eps scale: sum of per-row spreads, fixed order
        if (q == 0) spread[row] = valid ? (double)v.smax - (double)v.smin : 0.0;
        __syncthreads();
        for (int st = kBidRows / 2; st >= 1; st >>= 1) {
            if (tid < st) spread[tid] += spread[tid + st];
            __syncthreads();
        }
        if (tid == 0) W.part[blockIdx.x] = spread[0];
    }
}

// Round r, prices: one workgroup per cluster.  An over-full cluster finds the
// (m+1)-th largest margin in its list by a 4-pass radix select on the fp32
// bits (margins are >= 0, so bit order is value order; the list order does
// not matter) and raises its price by that margin plus eps_r; it also counts
// itself in flags[r & 1].  A list of up to kKmPriceLds margins is copied into
// LDS once and the passes read it there.  The eps scale (the round-0 spread
// sums, added in workgroup order) is formed in round 0 and kept in
// part[nbid].  Every workgroup clears its count for the next round.
constexpr int kKmPriceLds = 16384;

__global__ __launch_bounds__(kKmPriceThreads) void km_price_k(int n, int k, int m, int r,
                                                              int nbid, KmWork W) {
    constexpr int kBatch = 4;
    constexpr int kCopy = 8;
    static_assert(kKmPriceThreads == 256, "one thread per radix digit");
    __shared__ int hist[256];
    __shared__ int scan[8];
    __shared__ uint32_t s_pref;
    __shared__ int s_rank;
    __shared__ uint32_t sl[kKmPriceLds];
    const int j = blockIdx.x, tid = threadIdx.x;
    if (W.flags[2]) return;
    const int c = W.count[j];
    __syncthreads();
    if (tid == 0) W.count[j] = 0;
    if (c <= m) return;
    if (tid == 0) {
        s_pref = 0u;
        s_rank = m;  // 0-based rank from the top
    }
    const float *lst = W.list + (size_t)j * n;
    const bool inl = c <= kKmPriceLds;  // workgroup-uniform
    if (inl) {
        for (int i0 = 0; i0 < c; i0 += kCopy * kKmPriceThreads) {
            uint32_t v[kCopy];
#pragma unroll
            for (int u = 0; u < kCopy; ++u)
                v[u] = __float_as_uint(lst[min(i0 + u * kKmPriceThreads + tid, c - 1)]);
#pragma unroll
            for (int u = 0; u < kCopy; ++u)
                if (i0 + u * kKmPriceThreads + tid < c) sl[i0 + u * kKmPriceThreads + tid] = v[u];
        }
    }
    {
        uint32_t mask = 0u;
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            hist[tid] = 0;
            __syncthreads();
            const uint32_t pref = s_pref;
            for (int i0 = 0; i0 < c; i0 += kBatch * kKmPriceThreads) {
                uint32_t v[kBatch];
    #pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int ix = min(i0 + u * kKmPriceThreads + tid, c - 1);
                    v[u] = inl ? sl[ix] : __float_as_uint(lst[ix]);
                }
    #pragma unroll
                for (int u = 0; u < kBatch; ++u)
                    if (i0 + u * kKmPriceThreads + tid < c && (v[u] & mask) == pref)
                        atomicAdd(&hist[(v[u] >> shift) & 255], 1);
            }
            __syncthreads();
            {  // digits from the top: thread t takes digit 255 - t; the selected
               // digit is where the running count first exceeds the rank
                const int h = hist[255 - tid], rank = s_rank;
                int ex, ex1, tot, tot1;
                block_excl_scan2(h, 0, &ex, &ex1, &tot, &tot1, scan);
                __syncthreads();
                if (ex <= rank && rank < ex + h) {
                    s_rank = rank - ex;
                    s_pref = pref | ((uint32_t)(255 - tid) << shift);
                }
            }
            mask |= 255u << shift;
            __syncthreads();
        }
    }
    if (tid == 0) {
        double scale = 0.0;
        if (r == 0) {  // every over-full cluster forms the same value
            for (int b = 0; b < nbid; ++b) scale += W.part[b];
            scale /= (double)n;
            W.part[nbid] = scale;
        } else {
            scale = W.part[nbid];
        }
        double e = 0.3 * pow(0.9, (double)r);
        if (e < 0x1p-22) e = 0x1p-22;
        W.lam[j] += (double)__uint_as_float(s_pref) + e * scale;
        atomicAdd(&W.flags[r & 1], 1);
    }
}

// Edge row a of the shortest-path finish: base[a][b] = min over a's rows i
// of s_bi - s_ai and the row attaining it (lowest index on ties, so the
// member-list order does not matter); b = a and empty clusters give +inf.
// Wavefront w takes b = w, w + 16, ...; lanes stride over the members.
__device__ void ssp_row(const float *__restrict__ S, int n, int k, int a, int na,
                        const int32_t *memb, double *base, int32_t *bidx) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    for (int b = wv; b < k; b += kKmSspThreads / 64) {
        double best = INFINITY;
        int bi = 0x7FFFFFFF;
        if (b != a) {
            for (int t = lane; t < na; t += 64) {
                const int i = memb[(size_t)a * n + t];
                const double v = (double)S[(size_t)b * n + i] - (double)S[(size_t)a * n + i];
                if (v < best || (v == best && i < bi)) {
                    best = v;
                    bi = i;
                }
            }
        }
#pragma unroll
        for (int st = 32; st >= 1; st >>= 1) {
            const double ov = __shfl_xor(best, st, 64);
            const int oi = __shfl_xor(bi, st, 64);
            if (ov < best || (ov == best && oi < bi)) {
                best = ov;
                bi = oi;
            }
        }
        if (lane == 0) {
            base[(size_t)a * k + b] = best;
            bidx[(size_t)a * k + b] = bi;
        }
    }
}

// All edge rows at once, one workgroup per cluster, from the member lists of
// the bid round that precedes the finish (its argmax matches the prices).
__global__ __launch_bounds__(kKmSspThreads) void km_ssp_rows_k(const float *__restrict__ S, int n,
                                                               int k, KmWork W) {
    ssp_row(S, n, k, blockIdx.x, W.count[blockIdx.x], W.memb, W.base, W.bidx);
}

// Shortest-path finish of an assignment step (one workgroup; every loop is
// bounded by n, the largest possible excess).  Starts from the bid round's
// argmax assignment, counts and member lists, then per augmentation:
// multi-source Dijkstra from the over-full clusters over reduced costs
// max(0, base[u][v] + lambda_v - lambda_u) until the first under-full
// cluster t is settled; the path's rows move one edge each; lambda_v -=
// min(dist_v, dist_t); the edge rows of the clusters on the path are
// recomputed.  Sets flags[2] when balanced, flags[3] = augmentations, and
// clears the counts.
__global__ __launch_bounds__(kKmSspThreads) void km_ssp_k(const float *__restrict__ S, int n, int k,
                                                          int m, KmWork W,
                                                          int32_t *__restrict__ assign) {
    __shared__ double lam[kKmMaxK], dist[kKmMaxK];
    __shared__ int cnt[kKmMaxK], pred[kKmMaxK], settled[kKmMaxK], chg[kKmMaxK];
    __shared__ int s_u, s_t, s_excess;
    int32_t *memb = W.memb;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    for (int j = tid; j < k; j += kKmSspThreads) {
        lam[j] = W.lam[j];
        cnt[j] = W.count[j];
    }
    __syncthreads();
    int aug = 0;
    for (; aug <= n; ++aug) {
        if (wv == 0) {
            int ex = 0;
            for (int j = lane; j < k; j += 64) ex += cnt[j] > m ? cnt[j] - m : 0;
#pragma unroll
            for (int st = 32; st >= 1; st >>= 1) ex += __shfl_xor(ex, st, 64);
            if (lane == 0) s_excess = ex;
        }
        for (int v = tid; v < k; v += kKmSspThreads) {
            dist[v] = cnt[v] > m ? 0.0 : INFINITY;
            pred[v] = -1;
            settled[v] = 0;
            chg[v] = 0;
        }
        __syncthreads();
        if (s_excess == 0) break;
        // Dijkstra until the first under-full cluster is settled
        for (int step = 0; step < k; ++step) {
            if (wv == 0) {
                double bd = INFINITY;
                int bu = 0x7FFFFFFF;
                for (int v = lane; v < k; v += 64)
                    if (!settled[v] && (dist[v] < bd || (dist[v] == bd && v < bu))) {
                        bd = dist[v];
                        bu = v;
                    }
#pragma unroll
                for (int st = 32; st >= 1; st >>= 1) {
                    const double od = __shfl_xor(bd, st, 64);
                    const int ou = __shfl_xor(bu, st, 64);
                    if (od < bd || (od == bd && ou < bu)) {
                        bd = od;
                        bu = ou;
                    }
                }
                if (lane == 0) {
                    s_u = (bu < k && bd < INFINITY) ? bu : -1;
                    if (s_u >= 0) settled[s_u] = 1;
                    s_t = (s_u >= 0 && cnt[s_u] < m) ? s_u : -1;
                }
            }
            __syncthreads();
            const int u = s_u;
            if (u < 0 || s_t >= 0) break;
            for (int v = tid; v < k; v += kKmSspThreads) {
                if (settled[v]) continue;
                const double red = fmax(0.0, W.base[(size_t)u * k + v] + lam[v] - lam[u]);
                const double nd = dist[u] + red;
                if (nd < dist[v]) {
                    dist[v] = nd;
                    pred[v] = u;
                }
            }
            __syncthreads();
        }
        const int t = s_t;
        if (t < 0) break;  // no path: leaves flags[2] clear
        if (tid == 0) {  // move one row along each edge of the path, t back to its source
            for (int v = t, guard = 0; pred[v] >= 0 && guard < k; ++guard) {
                const int u = pred[v];
                const int p = W.bidx[(size_t)u * k + v];
                const int pu = W.pos[p], last = memb[(size_t)u * n + cnt[u] - 1];
                memb[(size_t)u * n + pu] = last;
                W.pos[last] = pu;
                memb[(size_t)v * n + cnt[v]] = p;
                W.pos[p] = cnt[v];
                --cnt[u];
                ++cnt[v];
                assign[p] = v;
                chg[u] = chg[v] = 1;
                v = u;
            }
        }
        __syncthreads();
        const double dt = dist[t];
        for (int v = tid; v < k; v += kKmSspThreads) lam[v] -= fmin(dist[v], dt);
        __syncthreads();
        for (int a = 0; a < k; ++a)
            if (chg[a]) ssp_row(S, n, k, a, cnt[a], memb, W.base, W.bidx);
        __syncthreads();
    }
    for (int j = tid; j < k; j += kKmSspThreads) {
        W.lam[j] = lam[j];
        W.count[j] = 0;
    }
    if (tid == 0) {
        W.flags[2] = s_excess == 0 ? 1 : 0;
        W.flags[3] = aug;
    }
}

// sum_i ||x_i - mu_a(i)||^2 = sum_i (||x_i||^2 + s_{a(i), i}), fp64, one
// workgroup, thread t takes rows t, t + 1024, ... then a fixed tree.
__global__ __launch_bounds__(1024) void km_objective_k(const float *__restrict__ S,
                                                       const double *__restrict__ xnorm,
                                                       const int32_t *__restrict__ assign, int n,
                                                       float *__restrict__ out) {
    __shared__ double red[1024];
    const int tid = threadIdx.x;
    double acc = 0.0;
    for (int i = tid; i < n; i += 1024) acc += xnorm[i] + (double)S[(size_t)assign[i] * n + i];
    red[tid] = acc;
    __syncthreads();
    for (int s = 512; s >= 1; s >>= 1) {
        if (tid < s) red[tid] += red[tid + s];
        __syncthreads();
    }
    if (tid == 0) *out = (float)red[0];
}

// Pi: cluster j's rows, ascending, at perm[j m ..].  One workgroup per
// cluster, a block scan over the rows in order.
__global__ __launch_bounds__(256) void km_perm_k(const int32_t *__restrict__ assign, int n, int m,
                                                 int32_t *__restrict__ perm) {
    __shared__ int scan[8];
    const int j = blockIdx.x, tid = threadIdx.x;
    int base = 0;
    for (int i0 = 0; i0 < n; i0 += 256) {
        const int i = i0 + tid;
        const int f = (i < n && assign[i] == j) ? 1 : 0;
        int ex, ex1, tot, tot1;
        block_excl_scan2(f, 0, &ex, &ex1, &tot, &tot1, scan);
        if (f && base + ex < m) perm[(size_t)j * m + base + ex] = i;
        base += tot;
    }
}

// mu_j[c] = mean over cluster j's rows (Pi order, fp64 sum), grid (k, D/256).
__global__ __launch_bounds__(256) void km_update_k(const uint16_t *__restrict__ F, int D, int m,
                                                   const int32_t *__restrict__ perm,
                                                   float *__restrict__ mu) {
    const int j = blockIdx.x, c = blockIdx.y * 256 + threadIdx.x;
    if (c >= D) return;
    double acc = 0.0;
    for (int t = 0; t < m; ++t) acc += bf16_to_f32(F[(size_t)perm[(size_t)j * m + t] * D + c]);
    mu[(size_t)j * D + c] = (float)(acc / (double)m);
}

__global__ void km_prices_out_k(const double *__restrict__ lam, int k, float *__restrict__ out) {
    for (int j = threadIdx.x; j < k; j += blockDim.x) out[j] = (float)lam[j];
}

template <int NT>
void launch_dist_nt(const uint16_t *F, int n, int D, int k, const KmWork &W, hipStream_t s) {
    const int blocks = (n + 16 * kKmDistWaves - 1) / (16 * kKmDistWaves);
    hipLaunchKernelGGL(km_dist_k<NT>, dim3(blocks), dim3(64 * kKmDistWaves), 0, s, F, n, D, k,
                       W.mu3, W.cn, W.S);
}

template <int... Q>
void launch_dist(int nt, const uint16_t *F, int n, int D, int k, const KmWork &W, hipStream_t s,
                 std::integer_sequence<int, Q...>) {
    ((nt == Q + 1 ? launch_dist_nt<Q + 1>(F, n, D, k, W, s) : void()), ...);
}

}  // namespace
}  // namespace pp

extern "C" size_t prunepath_kmeans_workspace(int32_t n, int32_t D, int32_t k) {
    if (k < 1 || k > pp::kKmMaxK || n < k || n > pp::kKmMaxN || n % k != 0) return 0;
    if (D < 64 || D > pp::kKmMaxD || D % 64 != 0) return 0;
    return pp::km_layout(n, D, k, nullptr, nullptr);
}

extern "C" pp_status prunepath_balanced_kmeans(const uint16_t *F, int32_t n, int32_t D, int32_t k,
                                               const float *init_centroids, int32_t iters,
                                               int32_t *assign, int32_t *perm, float *centroids,
                                               float *objective, float *prices, int32_t *rounds,
                                               void *workspace, void *hip_stream) {
    using namespace pp;
    if (!F || !init_centroids || !assign || !perm || !centroids || !workspace) return PP_EINVAL;
    if (prunepath_kmeans_workspace(n, D, k) == 0 || iters < 1 || iters > 1000) return PP_EINVAL;
    if ((reinterpret_cast<uintptr_t>(F) | reinterpret_cast<uintptr_t>(workspace)) & 15)
        return PP_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    KmWork W;
    km_layout(n, D, k, &W, static_cast<char *>(workspace));
    const int m = n / k, nbid = bid_blocks(n), nt = (k + 15) / 16;
    hipError_t e = hipSuccess;
    if (centroids != init_centroids)
        e = hipMemcpyAsync(centroids, init_centroids, sizeof(float) * (size_t)k * D,
                           hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return PP_EHIP;
    hipLaunchKernelGGL(km_xnorm_k, dim3((n + 3) / 4), dim3(256), 0, s, F, n, D, W.xnorm);
    pp_status status = PP_OK;
    for (int it = 0; it < iters && status == PP_OK; ++it) {
        hipLaunchKernelGGL(km_split_k, dim3(k), dim3(256), 0, s, centroids, k, D, W.mu3, W.cn);
        launch_dist(nt, F, n, D, k, W, s, std::make_integer_sequence<int, kKmMaxK / 16>{});
        hipLaunchKernelGGL(km_auction_init_k, dim3(1), dim3(256), 0, s, k, W.lam, W.count, W.flags);
        int r = 0, used = 0;
        bool done = false;
        while (!done && r < kKmAuctionRounds) {
            const int r1 = r + kKmBatch;
            for (; r < r1; ++r) {
                hipLaunchKernelGGL(km_bid_k, dim3(nbid), dim3(kKmBidThreads), 0, s, W.S, n, k, r,
                                   W, assign);
                hipLaunchKernelGGL(km_price_k, dim3(k), dim3(kKmPriceThreads), 0, s, n, k, m, r,
                                   nbid, W);
            }
            int32_t fl[4];
            if (hipMemcpyAsync(fl, W.flags, sizeof fl, hipMemcpyDeviceToHost, s) != hipSuccess ||
                hipStreamSynchronize(s) != hipSuccess)
                return PP_EHIP;
            // converged when a round left no cluster over-full: either a later
            // bid round saw it (done flag) or it was the last round enqueued
            done = fl[2] != 0 || fl[(r - 1) & 1] == 0;
            used = fl[2] != 0 ? fl[3] : r;
        }
        if (!done) {  // route the remaining excess by shortest paths
            // one more bid round: the argmax, counts and member lists of the
            // current prices (no price round follows it)
            hipLaunchKernelGGL(km_bid_k, dim3(nbid), dim3(kKmBidThreads), 0, s, W.S, n, k, r, W,
                               assign);
            hipLaunchKernelGGL(km_ssp_rows_k, dim3(k), dim3(kKmSspThreads), 0, s, W.S, n, k, W);
            hipLaunchKernelGGL(km_ssp_k, dim3(1), dim3(kKmSspThreads), 0, s, W.S, n, k, m, W,
                               assign);
            int32_t fl[4];
            if (hipMemcpyAsync(fl, W.flags, sizeof fl, hipMemcpyDeviceToHost, s) != hipSuccess ||
                hipStreamSynchronize(s) != hipSuccess)
                return PP_EHIP;
            done = fl[2] != 0;
            used = r + fl[3];
        }
        if (rounds) rounds[it] = done ? used : -1;
        if (!done) {
            status = PP_ENOTCONVERGED;
            break;
        }
        if (objective)
            hipLaunchKernelGGL(km_objective_k, dim3(1), dim3(1024), 0, s, W.S, W.xnorm, assign, n,
                               objective + it);
        hipLaunchKernelGGL(km_perm_k, dim3(k), dim3(256), 0, s, assign, n, m, perm);
        hipLaunchKernelGGL(km_update_k, dim3(k, (D + 255) / 256), dim3(256), 0, s, F, D, m, perm,
                           centroids);
    }
    if (prices) hipLaunchKernelGGL(km_prices_out_k, dim3(1), dim3(256), 0, s, W.lam, k, prices);
    if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) return PP_EHIP;
    return status;
}
