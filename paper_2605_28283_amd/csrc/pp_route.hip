// Router: Eq. (routing_logits) GEMV, Eq. (softmax_prob), the descending order
// pi, the cumulative mass C and the tau cut of Eq. (tau_thresh_activate).
//
// logits_k : one workgroup of 16 wavefronts per (16-token tile, 16-expert
//            tile).  Wavefront w accumulates its contiguous share of the K-steps
//            of d with bf16 MFMA; the 16 partial tiles are summed in wavefront
//            order, then g = (W_r x + b) * inv_temp is stored.  The summation
//            order depends on d only, never on T, so a token's logits are the
//            same bits in any batch: routing is batch-invariant.
// select_k : one wavefront per token.  pi orders experts by descending g,
//            equal g by ascending expert index (ordering g orders p: softmax is
//            monotone).  With e_i = exp(g_i - g_max), S = sum e and
//            C_i = (e_pi1 + ... + e_pii) / S:
//              nucleus: k = min{i : C_i >= tau}, all E if tau >= 1;
//              strict:  k = max(1, #{i < E : C_i < tau} + [tau > 1]).
//            The kept prefix is found by repeated wavefront arg-max (DPP /
//            permlane exchanges, no LDS traffic), one expert at a time, which
//            costs O(k); past kMaxIterative kept experts the token falls back
//            to a bitonic sort of all experts.  When every expert is kept
//            (tau >= 1 nucleus, tau > 1 strict) the order comes from the sort.
//            For a decode batch (T <= 64) each token also sets its bit in the
//            per-expert token masks (device-scope atomic OR) and the last token
//            to finish writes the batch plan: the union of kept experts, each
//            with its tokens and its first pair row.
// Deterministic: no floating-point atomics.
#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kRouteWaves = 16;
constexpr int kMaxIterative = 16;  // kept experts found by arg-max before falling back to a sort

struct RouteParams {
    const uint16_t *x;
    int T, d, E, NS;
    const uint16_t *Wr;
    const float *bias;
    const float *inv_temp;
    float tau;
    uint32_t flags;
    int nEt;
    float *glog;         // [T][E] logits
    int32_t *idx;
    int32_t *count;
    float *gate_w;
    uint32_t *selmask;
    float *gsig;
    PlanView plan;       // written when build_plan != 0
    int build_plan;
    unsigned long long *emask;  // [E] tokens of the batch that kept each expert (zero between calls)
    uint32_t *plan_cnt;         // arrival counter of the plan builder
};

__global__ __launch_bounds__(1024) void logits_k(RouteParams P) {
    __shared__ f32x4 red[kRouteWaves][64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int tt = blockIdx.x / P.nEt, et = blockIdx.x - tt * P.nEt;
    const int tr = tt * kRouteTile + (lane & 15);
    const int ec = et * kRouteTile + (lane & 15);
    const int koff = 8 * (lane >> 4);
    const bool va = tr < P.T, vb = ec < P.E;
    const uint16_t *xa = P.x + (size_t)(va ? tr : 0) * P.d + koff;
    const uint16_t *wb = P.Wr + (size_t)(vb ? ec : 0) * P.d + koff;
    const int spw = (P.NS + kRouteWaves - 1) / kRouteWaves;  // K-steps per wavefront (<= 16)
    const int s_lo = wv * spw, s_hi = min(P.NS, s_lo + spw);
    const uint4 z = make_uint4(0, 0, 0, 0);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int b0 = s_lo; b0 < s_hi; b0 += 8) {
        uint4 a[8], b[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int s = b0 + i;
            a[i] = (va && s < s_hi) ? ldg16(xa + s * kKStep) : z;
            b[i] = (vb && s < s_hi) ? ldg16(wb + s * kKStep) : z;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) acc = mfma16(a[i], b[i], acc);
    }
    red[wv][lane] = acc;
    __syncthreads();
    if (wv != 0) return;
    f32x4 r = red[0][lane];
#pragma unroll
    for (int w = 1; w < kRouteWaves; ++w) r += red[w][lane];
    // MFMA 16x16 result: lane holds rows 4*(lane/16)+i (tokens), column lane%16 (expert)
    if (!vb) return;
    const float bias = P.bias[ec];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int t = tt * kRouteTile + 4 * (lane >> 4) + i;
        if (t < P.T) {
            const float it = P.inv_temp ? P.inv_temp[t] : 1.0f;
            P.glog[(size_t)t * P.E + ec] = (r[i] + bias) * it;
        }
    }
}

// a comes before b in pi
__device__ __forceinline__ bool before(float ga, int ia, float gb, int ib) {
    return ga > gb || (ga == gb && ia < ib);
}

// Wavefront arg-max under `before`: every lane ends with the same (g, id).
__device__ __forceinline__ void wave_first(float &g, int &id, int lane) {
#pragma unroll
    for (int st = 1; st < 64; st <<= 1) {
        const float og = __uint_as_float(xor_lane_rt(__float_as_uint(g), st, lane));
        const int oi = (int)xor_lane_rt((uint32_t)id, st, lane);
        const bool take = before(og, oi, g, id);
        g = take ? og : g;
        id = take ? oi : id;
    }
}

// Sum over the wavefront of one value per lane, in one fixed order, returned
// identically to every lane.
__device__ __forceinline__ float wave_sum(float v) { return lane_value(wave_scan_f32(v), 63); }

// Full bitonic sort of (g, id) into pi order over 64*J lanes/registers.
template <int J>
__device__ __forceinline__ void sort_pi(float (&g)[J], int (&id)[J], int lane) {
    constexpr int N = 64 * J;
#pragma unroll
    for (int k = 2; k <= N; k <<= 1) {
#pragma unroll
        for (int st = k >> 1; st > 0; st >>= 1) {
            if (st >= 64) {
                const int js = st >> 6;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    if (j & js) continue;
                    const int jp = j | js;
                    const bool asc = ((j * 64 + lane) & k) == 0;
                    const bool sw = before(g[j], id[j], g[jp], id[jp]) != asc;
                    const float ga = g[j], gb = g[jp];
                    const int ia = id[j], ib = id[jp];
                    g[j] = sw ? gb : ga;
                    g[jp] = sw ? ga : gb;
                    id[j] = sw ? ib : ia;
                    id[jp] = sw ? ia : ib;
                }
            } else {
                const bool lower = (lane & st) == 0;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    const bool keep_first = lower == (((j * 64 + lane) & k) == 0);
                    const float og = __uint_as_float(xor_lane_rt(__float_as_uint(g[j]), st, lane));
                    const int oi = (int)xor_lane_rt((uint32_t)id[j], st, lane);
                    const bool sw = before(g[j], id[j], og, oi) != keep_first;
                    g[j] = sw ? og : g[j];
                    id[j] = sw ? oi : id[j];
                }
            }
        }
    }
}

// Output slot `pos` of token t holds expert e (kept) or nothing.
__device__ __forceinline__ void emit_slot(const RouteParams &P, int t, int pos, int e, float g,
                                          bool kept, uint32_t *sm) {
    const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
    const float w = sig ? 1.0f / (1.0f + expf(-g)) : 1.0f;
    P.idx[(size_t)t * P.E + pos] = kept ? e : -1;
    if (P.gate_w) P.gate_w[(size_t)t * P.E + pos] = kept ? w : 0.0f;
    if (kept) {
        P.gsig[(size_t)t * P.E + e] = w;
        atomicOr(&sm[e >> 5], 1u << (e & 31));
    }
}

// Records token t (< 64) in the per-expert masks of the decode plan.
__device__ __forceinline__ void mark_expert(const RouteParams &P, int t, int e) {
    __hip_atomic_fetch_or(P.emask + e, 1ull << t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Routes token t in one wavefront (the whole workgroup).
template <int J>
__device__ void route_token(const RouteParams &P, int t, int lane, uint32_t *sm, int *kept_e) {
    const float *lgt = P.glog + (size_t)t * P.E;
    const bool strict = (P.flags & PP_SELECT_STRICT) != 0;
    const bool all = strict ? (P.tau > 1.0f) : (P.tau >= 1.0f);
    float g[J];
    int id[J];
    float gmx = -INFINITY;
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const int e = lane + 64 * j;
        id[j] = e;
        g[j] = (e < P.E) ? lgt[e] : -INFINITY;
        gmx = fmaxf(gmx, g[j]);
    }
    // g_max and S = sum_i exp(g_i - g_max), identical on all lanes
#pragma unroll
    for (int st = 1; st < 64; st <<= 1)
        gmx = fmaxf(gmx, __uint_as_float(xor_lane_rt(__float_as_uint(gmx), st, lane)));
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < J; ++j) part += (id[j] < P.E) ? expf(g[j] - gmx) : 0.0f;
    const float S = wave_sum(part);
    if (lane < 8) sm[lane] = 0u;
    __builtin_amdgcn_wave_barrier();

    int k = 0;
    bool done = false;
    if (!all) {
        // repeated arg-max: the next expert of pi and its cumulative mass
        bool rm[J];
#pragma unroll
        for (int j = 0; j < J; ++j) rm[j] = id[j] >= P.E;
        float c = 0.0f;
        int m = 0;  // strict: #{i < E : C_i < tau} so far
        for (int pos = 0; pos < kMaxIterative && pos < P.E; ++pos) {
            float bg = -INFINITY;
            int bid = 0x7fffffff;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const bool tk = !rm[j] && before(g[j], id[j], bg, bid);
                bg = tk ? g[j] : bg;
                bid = tk ? id[j] : bid;
            }
            wave_first(bg, bid, lane);
#pragma unroll
            for (int j = 0; j < J; ++j) rm[j] = rm[j] || id[j] == bid;
            c += expf(bg - gmx);
            const float C = c / S;
            const bool below = pos < P.E - 1 && C < P.tau;
            bool keep, stop;
            if (strict) {
                keep = (pos == 0) || below;
                if (below) m = pos + 1;
                stop = !below;
            } else {
                keep = true;
                stop = (C >= P.tau) || (pos == P.E - 1);
            }
            if (keep && lane == 0) {
                emit_slot(P, t, pos, bid, bg, true, sm);
                kept_e[pos] = bid;
            }
            if (stop) {
                k = strict ? (m < 1 ? 1 : m) : pos + 1;
                done = true;
                break;
            }
        }
        if (done) {
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int pos = j * 64 + lane;
                if (pos >= k && pos < P.E) {
                    P.idx[(size_t)t * P.E + pos] = -1;
                    if (P.gate_w) P.gate_w[(size_t)t * P.E + pos] = 0.0f;
                }
            }
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
            if (P.build_plan && lane < k) mark_expert(P, t, kept_e[lane]);
        } else {
            // more than kMaxIterative kept experts: start over with a full sort
            __builtin_amdgcn_wave_barrier();
            if (lane < 8) sm[lane] = 0u;
            __builtin_amdgcn_wave_barrier();
        }
    }
    if (!done) {
        sort_pi<J>(g, id, lane);
        float cs[J];
        float carry = 0.0f;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const float ex = (id[j] < P.E) ? expf(g[j] - gmx) : 0.0f;
            cs[j] = wave_scan_f32(ex) + carry;
            carry = lane_value(cs[j], 63);
        }
        int mcount = 0;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int pos = j * 64 + lane;
            mcount += __popcll(__ballot(pos < P.E - 1 && cs[j] / S < P.tau));
        }
        if (strict) {
            k = mcount + (P.tau > 1.0f ? 1 : 0);
            k = k < 1 ? 1 : k;
        } else {
            k = all ? P.E : min(P.E, mcount + 1);
        }
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int pos = j * 64 + lane;
            if (pos < P.E) {
                emit_slot(P, t, pos, id[j], g[j], pos < k, sm);
                if (P.build_plan && pos < k) mark_expert(P, t, id[j]);
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    if (lane < 8) P.selmask[(size_t)t * 8 + lane] = sm[lane];
    if (lane == 0) P.count[t] = k;
}

// Decode plan for a batch of T <= 64 tokens, built by one wavefront from the
// per-expert token masks: groups = experts kept by at least one token
// (ascending expert index); group u owns pair rows [pair_u, pair_u + n_u),
// one per token, tokens ascending.  The masks are cleared for the next call.
__device__ void build_decode_plan(const RouteParams &P, int lane) {
    constexpr int kPer = kMaxExperts / 64;
    uint64_t m[kPer];
    int pc[kPer];
    int tot = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int e = lane * kPer + q;  // consecutive experts per lane keep the order ascending
        m[q] = e < P.E ? __hip_atomic_load(P.emask + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                       : 0ull;
        if (e < P.E && m[q]) P.emask[e] = 0ull;
        pc[q] = __popcll(m[q]);
        tot += m[q] != 0;
    }
    // exclusive prefixes over lanes of (groups, pairs)
    int pairs = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) pairs += pc[q];
    const int incl_g = wave_incl_scan(tot), incl_p = wave_incl_scan(pairs);
    int slot = incl_g - tot, poff = incl_p - pairs;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        if (!m[q]) continue;
        const int e = lane * kPer + q;
        P.plan.grp_e[slot] = e;
        P.plan.grp_pair[slot] = poff;
        P.plan.grp_n[slot] = pc[q];
        P.plan.grp_tok[slot] = poff;
        int r = 0;
        for (uint64_t mm = m[q]; mm; mm &= mm - 1) P.plan.toklist[poff + r++] = __builtin_ctzll(mm);
        ++slot;
        poff += pc[q];
    }
    if (lane == 63) {
        P.plan.head[0] = incl_g;
        P.plan.head[1] = incl_p;
    }
}

// One wavefront per token; with a decode plan the last token to finish
// builds it.
template <int J>
__global__ __launch_bounds__(64) void select_k(RouteParams P) {
    __shared__ uint32_t sm[8];
    __shared__ int kept_e[kMaxIterative];
    __shared__ int s_last;
    const int lane = threadIdx.x;
    route_token<J>(P, blockIdx.x, lane, sm, kept_e);
    if (!P.build_plan) return;
    if (!arrive_last(P.plan_cnt, (unsigned)P.T, &s_last)) return;
    build_decode_plan(P, lane);
}

}  // namespace

hipError_t launch_route(pp_layer *L, const uint16_t *x, int T, float tau, const float *inv_temp,
                        int32_t *idx, int32_t *count, float *gate_w, bool build_plan,
                        hipStream_t s) {
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
    P.glog = L->gpart;
    P.idx = idx;
    P.count = count;
    P.gate_w = gate_w;
    P.selmask = L->selmask;
    P.gsig = L->gsig;
    P.plan = plan_view(L, false);
    P.build_plan = (build_plan && T <= kDecodeTile) ? 1 : 0;
    P.emask = L->emask;
    P.plan_cnt = L->counters;  // the router's counter comes first
    const int nTt = (T + kRouteTile - 1) / kRouteTile;
    prof_mark(L, PP_KERNEL_ROUTE, s, true);
    hipLaunchKernelGGL(logits_k, dim3(nTt * P.nEt), dim3(1024), 0, s, P);
    if (dm.E <= 64)
        hipLaunchKernelGGL(select_k<1>, dim3(T), dim3(64), 0, s, P);
    else if (dm.E <= 128)
        hipLaunchKernelGGL(select_k<2>, dim3(T), dim3(64), 0, s, P);
    else
        hipLaunchKernelGGL(select_k<4>, dim3(T), dim3(64), 0, s, P);
    prof_mark(L, PP_KERNEL_ROUTE, s, false);
    return hipGetLastError();
}

}  // namespace pp
