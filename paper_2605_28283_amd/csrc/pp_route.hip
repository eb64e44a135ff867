// Fused router: Eq. (routing_logits) GEMV, Eq. (softmax_prob), the descending
// order pi, the cumulative mass C and the tau cut of Eq. (tau_thresh_activate).
//
// Grid: one workgroup (4 wavefronts) per (16-token tile, 16-expert tile,
// K-slice of 16 K-steps = 512 columns of d).  Each wavefront accumulates a 16x16 logit tile with bf16 MFMA over
// every fourth 32-wide K-step of the slice; the four tiles are summed in a
// fixed order and the slice's partial logits are stored.  The workgroup that
// completes a token tile last (arrival counter;
// device-scope stores/loads carry the other slices' partials) then routes its 16 tokens, four per
// wavefront, interleaved so the four dependency chains overlap:
//   g = (sum of partials in slice order + b) * inv_temp
//   bitonic sort of (g, expert) over 64*J lanes/registers: larger g first,
//   equal g by ascending expert index (ordering g orders p: softmax is monotone)
//   p = exp(g - g_max) / sum, inclusive prefix sums C in sorted order
//   m = #{i < E : C_i < tau} over the first E-1 positions, then
//   nucleus: k = E if tau >= 1 else min(E, m + 1);  strict: k = max(1, m + [tau > 1]).
// The result is deterministic: no floating-point atomics anywhere.
#include "pp_internal.h"

namespace pp {
namespace {

struct RouteParams {
    const uint16_t *x;
    int T, d, E, NS;
    const uint16_t *Wr;
    const float *bias;
    const float *inv_temp;
    float tau;
    uint32_t flags;
    int KSr, nEt;
    float *gpart;
    uint32_t *cnt;
    int32_t *idx;
    int32_t *count;
    float *gate_w;
    uint32_t *selmask;
    float *gsig;
};

// a comes before b in pi
__device__ __forceinline__ bool before(float ga, int ia, float gb, int ib) {
    return ga > gb || (ga == gb && ia < ib);
}

template <int J, int kTokPerWave>
__device__ void route_tokens(const RouteParams &P, int tt, int wv, int lane, uint32_t *smask,
                             const float (*lg)[kMaxExperts]) {
    constexpr int N = 64 * J;
    float g[kTokPerWave][J];
    int id[kTokPerWave][J];
    int tok[kTokPerWave];
    bool tv[kTokPerWave];
#pragma unroll
    for (int m = 0; m < kTokPerWave; ++m) {
        const int tl = wv + 4 * m;
        tok[m] = tt * kRouteTile + tl;
        tv[m] = tok[m] < P.T;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int e = lane + 64 * j;
            id[m][j] = e;
            g[m][j] = (tv[m] && e < P.E) ? lg[tl][e] : -INFINITY;
        }
    }
    bool any = false;
#pragma unroll
    for (int m = 0; m < kTokPerWave; ++m) any |= tv[m];
    if (!any) return;
    // bitonic sort, "smaller" = comes first in pi
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
#pragma unroll
                    for (int m = 0; m < kTokPerWave; ++m) {
                        const bool f = before(g[m][j], id[m][j], g[m][jp], id[m][jp]);
                        if (f != asc) {
                            float tg = g[m][j];
                            g[m][j] = g[m][jp];
                            g[m][jp] = tg;
                            int ti = id[m][j];
                            id[m][j] = id[m][jp];
                            id[m][jp] = ti;
                        }
                    }
                }
            } else {
                const bool lower = (lane & st) == 0;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    const bool asc = ((j * 64 + lane) & k) == 0;
#pragma unroll
                    for (int m = 0; m < kTokPerWave; ++m) {
                        const float og = __shfl_xor(g[m][j], st, 64);
                        const int oi = __shfl_xor(id[m][j], st, 64);
                        const bool f = before(g[m][j], id[m][j], og, oi);
                        if (f != (lower == asc)) {
                            g[m][j] = og;
                            id[m][j] = oi;
                        }
                    }
                }
            }
        }
    }
    const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
    const bool strict = (P.flags & PP_SELECT_STRICT) != 0;
#pragma unroll
    for (int m = 0; m < kTokPerWave; ++m) {
        const float gmax = __shfl(g[m][0], 0, 64);
        float ex[J];
        float part = 0.0f;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            ex[j] = (id[m][j] < P.E) ? expf(g[m][j] - gmax) : 0.0f;
            part += ex[j];
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o, 64);
        const float S = __shfl(part, 0, 64);
        float carry = 0.0f;
        int mcount = 0;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            float c = ex[j] / S;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const float n = __shfl_up(c, o, 64);
                if (lane >= o) c += n;
            }
            c += carry;
            carry = __shfl(c, 63, 64);
            const int pos = j * 64 + lane;
            mcount += __popcll(__ballot(pos < P.E - 1 && c < P.tau));
        }
        int k;
        if (strict) {
            k = mcount + (P.tau > 1.0f ? 1 : 0);
            k = k < 1 ? 1 : k;
        } else {
            k = (P.tau >= 1.0f) ? P.E : min(P.E, mcount + 1);
        }
        if (!tv[m]) continue;
        const int t = tok[m];
        if (lane < 8) smask[m * 8 + lane] = 0u;
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int pos = j * 64 + lane;
            const int e = id[m][j];
            if (pos < P.E) {
                const float w = sig ? 1.0f / (1.0f + expf(-g[m][j])) : 1.0f;
                P.idx[(size_t)t * P.E + pos] = pos < k ? e : -1;
                if (P.gate_w) P.gate_w[(size_t)t * P.E + pos] = pos < k ? w : 0.0f;
                if (e < P.E) P.gsig[(size_t)t * P.E + e] = w;
                if (pos < k && e < P.E) atomicOr(&smask[m * 8 + (e >> 5)], 1u << (e & 31));
            }
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
        if (lane < 8) P.selmask[(size_t)t * 8 + lane] = smask[m * 8 + lane];
        if (lane == 0) P.count[t] = k;
    }
}

template <int J>
__global__ __launch_bounds__(256) void route_k(RouteParams P) {
    __shared__ f32x4 red[4][64];
    __shared__ uint32_t smask[4][4 * 8];
    __shared__ int s_last;
    __shared__ float lg[kRouteTile][kMaxExperts];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int per_tile = P.nEt * P.KSr;
    const int tt = blockIdx.x / per_tile;
    const int rem = blockIdx.x % per_tile;
    const int et = rem / P.KSr, ks = rem % P.KSr;
    const int s0 = (int)((long)ks * P.NS / P.KSr), s1 = (int)((long)(ks + 1) * P.NS / P.KSr);
    const int tr = tt * kRouteTile + (lane & 15);
    const int ec = et * kRouteTile + (lane & 15);
    const int koff = 8 * (lane >> 4);
    const bool va = tr < P.T, vb = ec < P.E;
    const uint16_t *xa = P.x + (size_t)(va ? tr : 0) * P.d + koff;
    const uint16_t *wb = P.Wr + (size_t)(vb ? ec : 0) * P.d + koff;
    const uint4 z = make_uint4(0, 0, 0, 0);
    // a slice has at most kRouteSliceSteps = 16 K-steps: four per wavefront
    uint4 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int s = s0 + wv + 4 * i;
        const bool ok = s < s1;
        a[i] = (ok && va) ? ldg16(xa + s * kKStep) : z;
        b[i] = (ok && vb) ? ldg16(wb + s * kKStep) : z;
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) acc = mfma16(a[i], b[i], acc);
    red[wv][lane] = acc;
    __syncthreads();
    if (wv == 0) {
        f32x4 r = red[0][lane];
        r += red[1][lane];
        r += red[2][lane];
        r += red[3][lane];
        // MFMA 16x16 result: lane holds rows 4*(lane/16)+i (tokens), column lane%16 (expert)
        const int e = et * kRouteTile + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int t = tt * kRouteTile + 4 * (lane >> 4) + i;
            if (t < P.T && e < P.E) st_dev(P.gpart + ((size_t)ks * P.T + t) * P.E + e, r[i]);
        }
    }
    if (!arrive_last(&P.cnt[tt], (unsigned)per_tile, &s_last)) return;
    // logits of the tile's tokens: slices summed in slice order (fixed), then
    // bias and temperature; all loads of a batch are issued before any add
    const int nt = min(kRouteTile, P.T - tt * kRouteTile);
    const int n_el = nt * P.E;
    for (int base = 0; base < n_el; base += 4 * 256) {
        float v[4][kRouteMaxSlices];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = base + q * 256 + threadIdx.x;
            const bool ok = i < n_el;
            const int t = tt * kRouteTile + (ok ? i / P.E : 0), e = ok ? i % P.E : 0;
#pragma unroll
            for (int k = 0; k < kRouteMaxSlices; ++k)
                v[q][k] = (ok && k < P.KSr) ? ld_dev(P.gpart + ((size_t)k * P.T + t) * P.E + e)
                                            : 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = base + q * 256 + threadIdx.x;
            if (i < n_el) {
                float sum = 0.0f;
#pragma unroll
                for (int k = 0; k < kRouteMaxSlices; ++k)
                    if (k < P.KSr) sum += v[q][k];
                const int tl = i / P.E, e = i % P.E;
                const int t = tt * kRouteTile + tl;
                const float it = P.inv_temp ? P.inv_temp[t] : 1.0f;
                lg[tl][e] = (sum + P.bias[e]) * it;
            }
        }
    }
    __syncthreads();
    // four wavefronts share the tile's tokens
    const int tpw = (nt + 3) / 4;
    if (tpw == 1)
        route_tokens<J, 1>(P, tt, wv, lane, smask[wv], lg);
    else if (tpw == 2)
        route_tokens<J, 2>(P, tt, wv, lane, smask[wv], lg);
    else
        route_tokens<J, 4>(P, tt, wv, lane, smask[wv], lg);
}

}  // namespace

// The K-slices depend on d only, never on T, so a token's logits are summed
// in the same order whatever batch it arrives in (routing is batch-invariant:
// decode slices and one large prefill batch select identically).
int route_split(const pp_dims &dm, int T) {
    (void)T;
    const int ks = (dm.NS + kRouteSliceSteps - 1) / kRouteSliceSteps;
    return ks < 1 ? 1 : ks;
}

hipError_t launch_route(pp_layer *L, const uint16_t *x, int T, float tau, const float *inv_temp,
                        int32_t *idx, int32_t *count, float *gate_w, hipStream_t s) {
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
    P.KSr = route_split(dm, T);
    P.nEt = (dm.E + kRouteTile - 1) / kRouteTile;
    P.gpart = L->gpart;
    P.cnt = L->counters;  // route region comes first
    P.idx = idx;
    P.count = count;
    P.gate_w = gate_w;
    P.selmask = L->selmask;
    P.gsig = L->gsig;
    const int nTt = (T + kRouteTile - 1) / kRouteTile;
    const dim3 grid(nTt * P.nEt * P.KSr);
    prof_mark(L, PP_KERNEL_ROUTE, s, true);
    if (dm.E <= 64)
        hipLaunchKernelGGL(route_k<1>, grid, dim3(256), 0, s, P);
    else if (dm.E <= 128)
        hipLaunchKernelGGL(route_k<2>, grid, dim3(256), 0, s, P);
    else
        hipLaunchKernelGGL(route_k<4>, grid, dim3(256), 0, s, P);
    prof_mark(L, PP_KERNEL_ROUTE, s, false);
    return hipGetLastError();
}

}  // namespace pp
