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
#include "pp_select.h"

namespace pp {
namespace {

constexpr int kLgTiles = 4;       // 16-token tiles per logits workgroup


__global__ __launch_bounds__(1024) void logits_k(RouteParams P) {
    __shared__ uint4 xs[kLgTiles][kRouteWaves][64];  // [token tile][K-step][lane]: A fragments
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int tb = blockIdx.x / P.KSr, ks = blockIdx.x - tb * P.KSr;
    if (P.build_plan && blockIdx.x == 0 && tid < P.E) P.emask[tid] = 0ull;
    const int s_end = min(kRouteWaves, P.NS - ks * kRouteWaves);  // K-steps in this slice
    // wavefront wv < nEt: the router fragments of expert tile wv for the
    // slice, loaded first so that their round trip overlaps the token staging
    // (native vectors: an array of uint4 would not stay in registers; an
    // expert column past E reads a clamped row, and its products land only
    // in outputs that are never stored)
    const int ec = wv * kRouteTile + (lane & 15);
    const bool ve = ec < P.E;
    u32x4_t b[kRouteWaves];
    if (wv < P.nEt) {
        const u32x4_t *wr = reinterpret_cast<const u32x4_t *>(
            P.Wr + (size_t)min(ec, P.E - 1) * P.d + ks * kRouteWaves * kKStep + 8 * (lane >> 4));
        if (s_end == kRouteWaves) {  // a whole slice: one base, immediate offsets
#pragma unroll
            for (int s = 0; s < kRouteWaves; ++s) b[s] = wr[s * (kKStep / 8)];
        } else {
#pragma unroll
            for (int s = 0; s < kRouteWaves; ++s) b[s] = wr[min(s, s_end - 1) * (kKStep / 8)];
        }
    }
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
    // accumulated in order in the MFMA accumulators
    f32x4 acc[kLgTiles];
#pragma unroll
    for (int j = 0; j < kLgTiles; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (wv < P.nEt) {
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

template <int TPB>
__global__ __launch_bounds__(kSelThreads) void select_k(RouteParams P) {
    __shared__ SelLds<TPB> S;
    const SelOut r = select_tokens<TPB>(P, (int)blockIdx.x, S);
    select_store<TPB>(P, S, r);
}

}  // namespace

hipError_t launch_route(pp_layer *L, const uint16_t *x, int T, float tau, const float *inv_temp,
                        int32_t *idx, int32_t *count, float *gate_w, bool build_plan,
                        hipStream_t s, bool select) {
    const pp_dims &dm = L->dm;
    const RouteParams P = route_params(L, x, T, tau, inv_temp, idx, count, gate_w, build_plan);
    prof_mark(L, PP_KERNEL_ROUTE, s, true);
    if (T <= kDecodeTile) {
        const int nTt = (T + 15) / 16;
        hipLaunchKernelGGL(logits_small_k, dim3(nTt * P.nEt * P.KSr), dim3(64), 0, s, P);
    } else {
        const int nTb = (T + 16 * kLgTiles - 1) / (16 * kLgTiles);
        hipLaunchKernelGGL(logits_k, dim3(nTb * P.KSr), dim3(1024), 0, s, P);
    }
    // small batches: one token per workgroup (shortest latency); large ones:
    // four tokens of 128 threads per workgroup (one workgroup wave on the chip);
    // without `select` the caller's next kernel selects (single-token decode)
    if (select) {
        if (T > kDecodeTile && dm.E <= 128)
            hipLaunchKernelGGL(select_k<4>, dim3((T + 3) / 4), dim3(kSelThreads), 0, s, P);
        else
            hipLaunchKernelGGL(select_k<1>, dim3(T), dim3(kSelThreads), 0, s, P);
    }
    prof_mark(L, PP_KERNEL_ROUTE, s, false);
    return hipGetLastError();
}

}  // namespace pp
