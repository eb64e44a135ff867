// Token routing shared by the router kernels and the single-token decode
// gate/up kernel (which selects its token's experts itself): the parameters
// of a routing call and the per-token selection, Eq. (softmax_prob), the
// descending order pi and the tau cut of Eq. (tau_thresh_activate).
#pragma once
#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kRouteWaves = 16;  // K-steps per router slice (also wavefronts per logits workgroup)
constexpr int kMaxSlices = kMaxWidth / kKStep / kRouteWaves;  // K-slices of the largest d

struct RouteParams {
    const uint16_t *x;
    int T, d, E, NS;
    const uint16_t *Wr;
    const float *bias;
    const float *inv_temp;
    float tau;
    uint32_t flags;
    int nEt, KSr;
    float *gpart;        // [KSr][T][E] partial logits of the K-slices
    int32_t *idx;
    int32_t *count;
    float *gate_w;
    uint32_t *selmask;
    float *gsig;
    int build_plan;             // decode batch: record per-expert token masks
    unsigned long long *emask;  // [E] tokens of the batch that kept each expert
};

// A routing call's parameters (host side).
inline RouteParams route_params(pp_layer *L, const uint16_t *x, int T, float tau,
                                const float *inv_temp, int32_t *idx, int32_t *count,
                                float *gate_w, bool build_plan) {
    const pp_dims &dm = L->dm;
    RouteParams P;
    P.x = x;
    P.T = T;
    P.d = dm.d;
    P.E = dm.E;
    P.NS = dm.NS;
    P.Wr = L->Wr;
    P.bias = L->bias;
    P.inv_temp = inv_temp;
    P.tau = tau;
    P.flags = L->flags;
    P.nEt = (dm.E + kRouteTile - 1) / kRouteTile;
    P.KSr = (dm.NS + kRouteWaves - 1) / kRouteWaves;
    P.gpart = L->gpart;
    P.idx = idx;
    P.count = count;
    P.gate_w = gate_w;
    P.selmask = L->selmask;
    P.gsig = L->gsig;
    P.build_plan = (build_plan && T <= kDecodeTile) ? 1 : 0;
    P.emask = L->emask;
    return P;
}

// Sort key of expert i with logit g: a larger key comes first in pi (larger
// g first, equal g by ascending index).  -0 is folded into +0 so that equal
// logits compare equal; the index part makes every key distinct, so the
// ranks below are a permutation of 0..E-1 for any input.
__device__ __forceinline__ unsigned long long pi_key(float g, int i) {
    uint32_t u = __float_as_uint(g + 0.0f);
    u ^= (u >> 31) ? 0xFFFFFFFFu : 0x80000000u;
    return ((unsigned long long)u << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)i);
}

// Routes TPB tokens per workgroup of kSelThreads threads (kSelThreads / TPB
// threads per token, at least one per expert).
//   1. thread e < E: g_e = (sum of the K-slice partials in slice order + b_e)
//      * inv_temp; g_max by a max reduction; e_e = exp(g_e - g_max).
//   2. S = sum of e over the experts (lane order, then the wavefront sum).
//   3. rank_i = #{j before i in pi} and B_i = sum of e_j over j before i,
//      counted per (slice of j, i) -- kSelThreads / EP slices of j, each
//      summed in j order, by one thread per (slice, i) or one thread taking
//      several slices in turn -- then summed slice by slice.  C at position
//      rank_i + 1 is (B_i + e_i) / S and C before it is B_i / S.
//   4. nucleus: expert i is kept iff rank_i == 0 or B_i / S < tau (every
//      expert when tau >= 1), so k = #kept = min{i : C_i >= tau};
//      strict: m = #{i : rank_i < E - 1, (B_i + e_i) / S < tau},
//      k = max(1, m + [tau > 1]); top-k: k = round(tau) in [1, E];
//      LTE: k = #{i : sigmoid(g_i) > tau}.  Kept iff rank_i < k.
// Floating-point addition is monotone, so B grows with the rank and the kept
// set is always a prefix of pi.  The work is O(E^2) per token with no
// dependence on k; all orders of summation are fixed and the same for every
// TPB, so a token's selection does not depend on T or on the launch.
constexpr int kSelThreads = 512;

// Sum over the wavefront of one value per lane, in one fixed order, returned
// identically to every lane.
__device__ __forceinline__ float wave_sum(float v) { return lane_value(wave_scan_f32(v), 63); }

// Steps 1-4 above for the TPB tokens of block `blk` (token blk * TPB + u),
// with kSelThreads threads; the scratch sc is this workgroup's LDS.  Returns
// the thread's view: its token and, for thread tt < E, the rank of expert tt
// in pi, the token's kept count k and sigmoid(g_tt).
struct SelOut {
    int u, tt, t;
    bool live;
    int rank, k;
    float sg;
};

template <int TPB>
struct SelLds {
    uint4 kk[TPB][kMaxExperts];  // (key lo, key hi, e bits, -)
    float2 part[TPB][kSelThreads];
    float wmax[kSelThreads / 64];
    uint32_t sm[TPB][8];
    int kc[TPB];
};

template <int TPB>
__device__ __forceinline__ SelOut select_tokens(const RouteParams &P, int blk, SelLds<TPB> &sc) {
    constexpr int TH = kSelThreads / TPB;  // threads per token
    constexpr int WPT = TH / 64;           // wavefronts per token
    static_assert(TH % 64 == 0, "whole wavefronts per token");
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int u = tid / TH, tt = tid - u * TH;  // token of the block, thread of the token
    const int t = blk * TPB + u;
    const bool live = t < P.T;
    const int tc = live ? t : P.T - 1;
    const int E = P.E;
    const bool strict = (P.flags & PP_SELECT_STRICT) != 0;
    const bool all = strict ? (P.tau > 1.0f) : (P.tau >= 1.0f);
    if (tt < 8) sc.sm[u][tt] = 0u;
    if (tt == 0) sc.kc[u] = 0;
    // 1. logits (all partial loads issued before the sum)
    float g = -INFINITY;
    if (tt < E) {
        float v[kMaxSlices];
#pragma unroll
        for (int k = 0; k < kMaxSlices; ++k)
            v[k] = P.gpart[((size_t)min(k, P.KSr - 1) * P.T + tc) * E + tt];
        const float b = P.bias[tt];
        const float it = P.inv_temp ? P.inv_temp[tc] : 1.0f;
        float sum = 0.0f;
#pragma unroll
        for (int k = 0; k < kMaxSlices; ++k)
            if (k < P.KSr) sum += v[k];
        g = (sum + b) * it;
    }
    float m = g;
#pragma unroll
    for (int st = 1; st < 64; st <<= 1)
        m = fmaxf(m, __uint_as_float(xor_lane_rt(__float_as_uint(m), st, lane)));
    if (lane == 0) sc.wmax[wv] = m;
    __syncthreads();
    float gmax = sc.wmax[u * WPT];
#pragma unroll
    for (int w = 1; w < WPT; ++w) gmax = fmaxf(gmax, sc.wmax[u * WPT + w]);
    const float ex = (tt < E) ? expf(g - gmax) : 0.0f;
    const unsigned long long key = pi_key(g, tt);
    // entries past E are zero keys, which come after every expert
    const int EP = E <= 64 ? 64 : (E <= 128 ? 128 : 256);
    if (tt < EP)
        sc.kk[u][tt] = tt < E ? make_uint4((uint32_t)key, (uint32_t)(key >> 32), __float_as_uint(ex), 0u)
                           : make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    // 2. S, computed the same way by every wavefront
    float sl = 0.0f;
    for (int i = lane; i < E; i += 64) sl += __uint_as_float(sc.kk[u][i].z);
    const float S = wave_sum(sl);
    // 3. ranks and preceding mass: (slice q of j, i) for q < nsl, i < EP
    const int nsl = kSelThreads / EP;
    {
        const int i = tt & (EP - 1);
        // slice of j: [q per, q per + per), per a multiple of 4; the slices
        // cover 0..E-1 and stay inside the EP entries of kk
        const int per = (((E + nsl - 1) / nsl) + 3) & ~3;
        const int tq = TH >= EP ? TH / EP : 1;  // threads per expert: slices q = tt / EP + tq r
        const unsigned long long ki =
            i < E ? (((unsigned long long)sc.kk[u][i].y << 32) | sc.kk[u][i].x) : 0ull;
        for (int q = tt / EP; q < nsl; q += tq) {
            float bm = 0.0f;
            int cnt = 0;
            if (i < E) {
                for (int j = q * per; j < q * per + per; j += 4) {
                    uint4 o[4];
#pragma unroll
                    for (int w = 0; w < 4; ++w) o[w] = sc.kk[u][j + w];
                    // keep the masses unconditional loads, issued with the
                    // keys: left to itself the compiler reloads one under its
                    // comparison (a branch and a second LDS round trip)
                    asm volatile("" : "+v"(o[0].z), "+v"(o[1].z), "+v"(o[2].z), "+v"(o[3].z));
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const bool bef = (((unsigned long long)o[w].y << 32) | o[w].x) > ki;
                        bm += bef ? __uint_as_float(o[w].z) : 0.0f;
                        cnt += bef ? 1 : 0;
                    }
                }
            }
            sc.part[u][q * EP + i] = make_float2(bm, __int_as_float(cnt));
        }
    }
    __syncthreads();
    // 4. the tau cut
    float B = 0.0f;
    int rank = 0;
    if (tt < E) {
        for (int q = 0; q < nsl; ++q) {
            const float2 pq = sc.part[u][q * EP + tt];
            B += pq.x;
            rank += __float_as_int(pq.y);
        }
    }
    const bool topk = (P.flags & PP_SELECT_TOPK) != 0;
    const bool lte = (P.flags & PP_SELECT_LTE) != 0;
    const float sg = 1.0f / (1.0f + expf(-g));  // sigmoid(g_e): LTE score and gate
    int cond = 0;
    if (tt < E) {
        if (lte)
            cond = sg > P.tau ? 1 : 0;
        else if (strict)
            cond = (rank < E - 1 && (B + ex) / S < P.tau) ? 1 : 0;
        else
            cond = (all || rank == 0 || B / S < P.tau) ? 1 : 0;
    }
    {
        const int wc = __popcll(__ballot(cond));
        if (lane == 0) atomicAdd(&sc.kc[u], wc);
    }
    __syncthreads();
    int k = sc.kc[u];
    if (topk) {
        k = (int)fminf(floorf(P.tau + 0.5f), (float)E);
        k = k < 1 ? 1 : k;
    } else if (strict) {
        k += P.tau > 1.0f ? 1 : 0;
        k = k < 1 ? 1 : k;
    }
    SelOut r;
    r.u = u;
    r.tt = tt;
    r.t = t;
    r.live = live;
    r.rank = rank;
    r.k = k;
    r.sg = sg;
    return r;
}

// Step 5: slot rank_i of token t holds expert i if kept, else nothing; the
// kept experts' gate weights, the token's kept-expert bitmask and count, and
// for a decode batch the per-expert token masks.
template <int TPB>
__device__ __forceinline__ void select_store(const RouteParams &P, SelLds<TPB> &sc,
                                             const SelOut &r) {
    const int u = r.u, tt = r.tt, t = r.t, E = P.E, rank = r.rank, k = r.k;
    const bool live = r.live;
    const float sg = r.sg;
    if (tt < E && live) {
        const bool kept = rank < k;
        const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
        const float w = sig ? sg : 1.0f;
        P.idx[(size_t)t * E + rank] = kept ? tt : -1;
        if (P.gate_w) P.gate_w[(size_t)t * E + rank] = kept ? w : 0.0f;
        if (kept) {
            P.gsig[(size_t)t * E + tt] = w;
            atomicOr(&sc.sm[u][tt >> 5], 1u << (tt & 31));
            if (P.build_plan)
                __hip_atomic_fetch_or(P.emask + tt, 1ull << t, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __syncthreads();
    if (tt < 8 && live) P.selmask[(size_t)t * 8 + tt] = sc.sm[u][tt];
    if (tt == 0 && live) P.count[t] = k;
}

}  // namespace
}  // namespace pp
