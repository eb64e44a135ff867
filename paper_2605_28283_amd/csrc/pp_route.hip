// Router: Eq. (routing_logits) GEMV, Eq. (softmax_prob), the descending order
// pi, the cumulative mass C and the tau cut of Eq. (tau_thresh_activate).
//
// logits_k : one workgroup per (64-token block, K-slice of 16 K-steps = 512
//            columns of d).  The block's token rows are staged in LDS as MFMA
//            operands; wavefront w takes expert tile w (16 experts) for all
//            four token tiles and accumulates the slice's 16 K-steps in order
//            in the MFMA accumulators (bf16 MFMA 16x16x32, fp32), storing the
//            slice's partial logits, staged in LDS and written as whole rows.
//            select_k sums the slices in slice order.
//            Every logit is formed in an order that depends on d only, never on
//            T or on the other tokens, so a token's logits are the same bits in
//            any batch: routing is batch-invariant.  Batches of up to 64 tokens
//            use logits_small_k (one wavefront per token tile x expert tile x
//            slice, the same MFMA chain).
// select_k : one token per workgroup (four per workgroup for batches past 64
//            tokens with E <= 128; the same sums).  pi orders experts by descending g,
//            equal g by ascending expert index (ordering g orders p: softmax is
//            monotone).  With e_i = exp(g_i - g_max), S = sum e and
//            C_i = (e_pi1 + ... + e_pii) / S:
//              nucleus: k = min{i : C_i >= tau}, all E if tau >= 1;
//              strict:  k = max(1, #{i < E : C_i < tau} + [tau > 1]).
//            Instead of sorting, each expert's rank in pi and the mass in
//            front of it are counted against all other experts (O(E^2) work
//            spread over the workgroup, independent of k), which gives every
//            C_i and the slot of each kept expert directly.  For a decode
//            batch (T <= 64) each kept expert also gets the token's bit in its
//            per-expert token mask (device-scope atomic OR); the gate/up
//            kernel derives the batch plan from them.
// Deterministic: no floating-point atomics.
#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kRouteWaves = 16;  // K-steps per slice (also wavefronts per logits workgroup)
constexpr int kLgTiles = 4;       // 16-token tiles per logits workgroup
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

__global__ __launch_bounds__(1024) void logits_k(RouteParams P) {
    __shared__ uint4 xs[kLgTiles][kRouteWaves][64];  // [token tile][K-step][lane]: A fragments
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int tb = blockIdx.x / P.KSr, ks = blockIdx.x - tb * P.KSr;
    if (P.build_plan && blockIdx.x == 0 && tid < P.E) P.emask[tid] = 0ull;
    const int s_end = min(kRouteWaves, P.NS - ks * kRouteWaves);  // K-steps in this slice
    // stage the block's token rows of this slice as MFMA A fragments; every
    // load is issued (addresses clamped into the operands), then rows past T
    // and K-steps past the slice are zeroed
    {
        const int s = wv, sc = min(s, s_end - 1);  // thread (wv, lane) stages K-step wv of every tile
        u32x4_t v[kLgTiles];  // native vectors: the selects below stay in registers
#pragma unroll
        for (int j = 0; j < kLgTiles; ++j) {
            const int t = min(tb * 16 * kLgTiles + 16 * j + (lane & 15), P.T - 1);
            v[j] = *reinterpret_cast<const u32x4_t *>(P.x + (size_t)t * P.d +
                                                      (ks * kRouteWaves + sc) * kKStep + 8 * (lane >> 4));
        }
#pragma unroll
        for (int j = 0; j < kLgTiles; ++j) {
            const int t = tb * 16 * kLgTiles + 16 * j + (lane & 15);
            const u32x4_t w = (t < P.T && s < s_end) ? v[j] : u32x4_t{0u, 0u, 0u, 0u};
            xs[j][s][lane] = make_uint4(w.x, w.y, w.z, w.w);
        }
    }
    __syncthreads();
    // wavefront wv: expert tile wv for every token tile, K-steps of the slice
    // accumulated in order in the MFMA accumulators; the slice's router
    // fragments are all loaded first
    const int ec = wv * kRouteTile + (lane & 15);
    const bool ve = ec < P.E;
    f32x4 acc[kLgTiles];
#pragma unroll
    for (int j = 0; j < kLgTiles; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (wv < P.nEt) {
        // (native vectors: an array of uint4 would not stay in registers; an
        // expert column past E reads a clamped row, and its products land only
        // in outputs that are never stored)
        u32x4_t b[kRouteWaves];
        const u32x4_t *wr = reinterpret_cast<const u32x4_t *>(
            P.Wr + (size_t)min(ec, P.E - 1) * P.d + ks * kRouteWaves * kKStep + 8 * (lane >> 4));
        if (s_end == kRouteWaves) {  // a whole slice: one base, immediate offsets
#pragma unroll
            for (int s = 0; s < kRouteWaves; ++s) b[s] = wr[s * (kKStep / 8)];
        } else {
#pragma unroll
            for (int s = 0; s < kRouteWaves; ++s) b[s] = wr[min(s, s_end - 1) * (kKStep / 8)];
        }
        const int ntile = min(kLgTiles, (P.T - tb * 16 * kLgTiles + 15) / 16);
        // two token tiles at a time (register budget), K-steps in order
#pragma unroll
        for (int j0 = 0; j0 < kLgTiles; j0 += 2) {
            if (j0 < ntile) {
#pragma unroll
                for (int s = 0; s < kRouteWaves; ++s) {
                    if (s < s_end) {
                        const uint4 bs = make_uint4(b[s].x, b[s].y, b[s].z, b[s].w);
                        acc[j0] = mfma16(xs[j0][s][lane], bs, acc[j0]);
                        if (j0 + 1 < ntile) acc[j0 + 1] = mfma16(xs[j0 + 1][s][lane], bs, acc[j0 + 1]);
                    }
                }
            }
        }
    }
    // the block's partial logits are one contiguous [rows][E] range of the
    // slice: staged in LDS (lane holds tokens 4 (lane / 16) + i of each tile,
    // expert ec), then written out with whole-row stores
    __syncthreads();
    float *ob = reinterpret_cast<float *>(&xs[0][0][0]);
    static_assert(sizeof(xs) >= 16 * kLgTiles * kMaxExperts * sizeof(float), "staging fits");
    if (wv < P.nEt && ve) {
#pragma unroll
        for (int j = 0; j < kLgTiles; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) ob[(16 * j + 4 * (lane >> 4) + i) * P.E + ec] = acc[j][i];
    }
    __syncthreads();
    const int t0 = tb * 16 * kLgTiles, rows = min(16 * kLgTiles, P.T - t0);
    float *dst = P.gpart + ((size_t)ks * P.T + t0) * P.E;
    const int n = rows * P.E;
    if (P.E % 4 == 0) {
        for (int i = tid; 4 * i < n; i += blockDim.x)
            reinterpret_cast<float4 *>(dst)[i] = reinterpret_cast<const float4 *>(ob)[i];
    } else {
        for (int i = tid; i < n; i += blockDim.x) dst[i] = ob[i];
    }
}

// The same arithmetic for small batches, with more parallelism: one
// wavefront per (16-token tile, 16-expert tile, K-slice), operands straight
// from memory.  Each partial logit is the same chain of MFMAs as in logits_k,
// so both kernels give identical bits.
__global__ __launch_bounds__(64) void logits_small_k(RouteParams P) {
    const int lane = threadIdx.x;
    const int per_tile = P.nEt * P.KSr;
    const int tt = blockIdx.x / per_tile;
    const int rem = blockIdx.x - tt * per_tile;
    const int et = rem / P.KSr, ks = rem - et * P.KSr;
    if (P.build_plan && blockIdx.x == 0) {
        for (int e = lane; e < P.E; e += 64) P.emask[e] = 0ull;
    }
    const int s_end = min(kRouteWaves, P.NS - ks * kRouteWaves);
    const int t = tt * 16 + (lane & 15), ec = et * kRouteTile + (lane & 15);
    const bool vt = t < P.T, ve = ec < P.E;
    const uint4 z = make_uint4(0, 0, 0, 0);
    const size_t col0 = (size_t)ks * kRouteWaves * kKStep + 8 * (lane >> 4);
    uint4 a[kRouteWaves], b[kRouteWaves];
#pragma unroll
    for (int s = 0; s < kRouteWaves; ++s) {
        a[s] = (vt && s < s_end) ? ldg16(P.x + (size_t)t * P.d + col0 + s * kKStep) : z;
        b[s] = (ve && s < s_end) ? ldg16(P.Wr + (size_t)ec * P.d + col0 + s * kKStep) : z;
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < kRouteWaves; ++s)
        if (s < s_end) acc = mfma16(a[s], b[s], acc);
    if (!ve) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int tr = tt * 16 + 4 * (lane >> 4) + i;
        if (tr < P.T) P.gpart[((size_t)ks * P.T + tr) * P.E + ec] = acc[i];
    }
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

template <int TPB>
__global__ __launch_bounds__(kSelThreads) void select_k(RouteParams P) {
    constexpr int TH = kSelThreads / TPB;  // threads per token
    constexpr int WPT = TH / 64;           // wavefronts per token
    static_assert(TH % 64 == 0, "whole wavefronts per token");
    __shared__ uint4 kk[TPB][kMaxExperts];  // (key lo, key hi, e bits, -)
    __shared__ float2 part[TPB][kSelThreads];
    __shared__ float wmax[kSelThreads / 64];
    __shared__ uint32_t sm[TPB][8];
    __shared__ int kc[TPB];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int u = tid / TH, tt = tid - u * TH;  // token of the block, thread of the token
    const int t = blockIdx.x * TPB + u;
    const bool live = t < P.T;
    const int tc = live ? t : P.T - 1;
    const int E = P.E;
    const bool strict = (P.flags & PP_SELECT_STRICT) != 0;
    const bool all = strict ? (P.tau > 1.0f) : (P.tau >= 1.0f);
    if (tt < 8) sm[u][tt] = 0u;
    if (tt == 0) kc[u] = 0;
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
    if (lane == 0) wmax[wv] = m;
    __syncthreads();
    float gmax = wmax[u * WPT];
#pragma unroll
    for (int w = 1; w < WPT; ++w) gmax = fmaxf(gmax, wmax[u * WPT + w]);
    const float ex = (tt < E) ? expf(g - gmax) : 0.0f;
    const unsigned long long key = pi_key(g, tt);
    // entries past E are zero keys, which come after every expert
    const int EP = E <= 64 ? 64 : (E <= 128 ? 128 : 256);
    if (tt < EP)
        kk[u][tt] = tt < E ? make_uint4((uint32_t)key, (uint32_t)(key >> 32), __float_as_uint(ex), 0u)
                           : make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    // 2. S, computed the same way by every wavefront
    float sl = 0.0f;
    for (int i = lane; i < E; i += 64) sl += __uint_as_float(kk[u][i].z);
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
            i < E ? (((unsigned long long)kk[u][i].y << 32) | kk[u][i].x) : 0ull;
        for (int q = tt / EP; q < nsl; q += tq) {
            float bm = 0.0f;
            int cnt = 0;
            if (i < E) {
                for (int j = q * per; j < q * per + per; j += 4) {
                    uint4 o[4];
#pragma unroll
                    for (int w = 0; w < 4; ++w) o[w] = kk[u][j + w];
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
            part[u][q * EP + i] = make_float2(bm, __int_as_float(cnt));
        }
    }
    __syncthreads();
    // 4. the tau cut
    float B = 0.0f;
    int rank = 0;
    if (tt < E) {
        for (int q = 0; q < nsl; ++q) {
            const float2 pq = part[u][q * EP + tt];
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
        if (lane == 0) atomicAdd(&kc[u], wc);
    }
    __syncthreads();
    int k = kc[u];
    if (topk) {
        k = (int)fminf(floorf(P.tau + 0.5f), (float)E);
        k = k < 1 ? 1 : k;
    } else if (strict) {
        k += P.tau > 1.0f ? 1 : 0;
        k = k < 1 ? 1 : k;
    }
    // 5. outputs: slot rank_i of token t holds expert i if kept, else nothing
    if (tt < E && live) {
        const bool kept = rank < k;
        const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
        const float w = sig ? sg : 1.0f;
        P.idx[(size_t)t * E + rank] = kept ? tt : -1;
        if (P.gate_w) P.gate_w[(size_t)t * E + rank] = kept ? w : 0.0f;
        if (kept) {
            P.gsig[(size_t)t * E + tt] = w;
            atomicOr(&sm[u][tt >> 5], 1u << (tt & 31));
            if (P.build_plan)
                __hip_atomic_fetch_or(P.emask + tt, 1ull << t, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __syncthreads();
    if (tt < 8 && live) P.selmask[(size_t)t * 8 + tt] = sm[u][tt];
    if (tt == 0 && live) P.count[t] = k;
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
    P.KSr = (dm.NS + kRouteWaves - 1) / kRouteWaves;
    P.gpart = L->gpart;
    P.idx = idx;
    P.count = count;
    P.gate_w = gate_w;
    P.selmask = L->selmask;
    P.gsig = L->gsig;
    P.build_plan = (build_plan && T <= kDecodeTile) ? 1 : 0;
    P.emask = L->emask;
    prof_mark(L, PP_KERNEL_ROUTE, s, true);
    if (T <= kDecodeTile) {
        const int nTt = (T + 15) / 16;
        hipLaunchKernelGGL(logits_small_k, dim3(nTt * P.nEt * P.KSr), dim3(64), 0, s, P);
    } else {
        const int nTb = (T + 16 * kLgTiles - 1) / (16 * kLgTiles);
        hipLaunchKernelGGL(logits_k, dim3(nTb * P.KSr), dim3(1024), 0, s, P);
    }
    // small batches: one token per workgroup (shortest latency); large ones:
    // four tokens of 128 threads per workgroup (one workgroup wave on the chip)
    if (T > kDecodeTile && dm.E <= 128)
        hipLaunchKernelGGL(select_k<4>, dim3((T + 3) / 4), dim3(kSelThreads), 0, s, P);
    else
        hipLaunchKernelGGL(select_k<1>, dim3(T), dim3(kSelThreads), 0, s, P);
    prof_mark(L, PP_KERNEL_ROUTE, s, false);
    return hipGetLastError();
}

}  // namespace pp
