// Decode expert evaluation (T <= 64): Eq. (ffn) restricted to the batch's
// kept experts and summed per token, Eqs. (moefication_decomp), (moe_output).
//
// The plan has one group per expert kept by at least one token of the batch:
// every gate/up workgroup derives it from the router's per-expert token masks
// and workgroup 0 stores it for the down projection.
//
//   gateup_dec_k: unit = (group, K-slice), the gate/up projections and the
//                 SiLU product of one group (code shared with prefill); the
//                 K-split is chosen so that all units fit in one round of
//                 resident workgroups.
//   down_dec_k  : unit = (64 rows of d, chunk of groups); each wavefront takes
//                 every fourth group of the chunk, multiplies its 64x128 down
//                 block with the group's compact token tiles (two MFMAs per
//                 fragment: hi and lo) and adds the result into its own LDS
//                 accumulator [tokens][64 rows] -- no synchronisation inside
//                 the chunk; the next half-group's fragments are loaded while
//                 the current one is multiplied.  The four accumulators are
//                 summed in wavefront order; chunks are summed in chunk order by
//                 the last to arrive.  No float atomics: decode is deterministic.
#include "pp_gateup.h"

namespace pp {
namespace {

constexpr int kDnRows = 64;        // rows of d per down unit
constexpr int kMaxChunks = 32;     // expert chunks per row block, at most
constexpr int kDnMinPerChunk = 8;  // groups per chunk at least (two per wavefront)

struct DNParams {
    int T, d, E;
    const uint16_t *Wd;
    const uint16_t *h_hi;
    const uint16_t *h_lo;
    float *y;
    float *ypart;
    size_t ypart_elems;
    uint32_t *cnt;
    PlanView plan;
};

// ------------------------------------------------------------------ gate/up

__global__ __launch_bounds__(kGuThreads, 4) void gateup_dec_k(GUParams P) {
    __shared__ uint4 xf[kXBufBytes / 16];
    __shared__ int stok[kGroupTokens];
    __shared__ int s_flag;
    __shared__ DecodePlan D;
    const int tid = threadIdx.x;
    decode_plan<true>(P, D);
    const int nG = D.nG, npairs = D.npairs;
    const int KS = choose_ks(P, nG, npairs, (int)gridDim.x);
    const int units = nG * KS;
    for (int unit = (int)blockIdx.x; unit < units; unit += (int)gridDim.x) {
        const int g = unit / KS, ks = unit - g * KS;
        const unsigned long long m = D.mask[g];
        if (tid < 64 && ((m >> tid) & 1ull)) stok[__popcll(m & ((1ull << tid) - 1ull))] = tid;
        __syncthreads();
        gateup_group(P, D.e[g], __popcll(m), D.pair[g], g, ks, KS, npairs, stok, xf,
                            &s_flag);
        __syncthreads();
    }
}

// ------------------------------------------------------------------ down

// Half of one expert's decode down work, as held in registers by a
// wavefront: 32 rows of its 64-row down block (2 row tiles x 4 K-steps of A
// fragments) and the B fragments (h hi and lo) of its first 16 tokens.
struct DownItem {
    uint4 w[2][4];
    uint4 bh[4], bl[4];
    int tok, n, p0, tk, half;
};

__device__ __forceinline__ void load_down_item(const DNParams &P, int u, int half, int rb, int RT,
                                               int lane, DownItem &it) {
    const uint4 z = make_uint4(0, 0, 0, 0);
    const int e = P.plan.grp_e[u];
    it.n = P.plan.grp_n[u];
    it.p0 = P.plan.grp_pair[u];
    it.tk = P.plan.grp_tok[u];
    it.half = half;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
        const uint16_t *wp =
            P.Wd + (((size_t)e * RT + rb * 4 + 2 * half + mt) * 4 * 64 + lane) * 8;
#pragma unroll
        for (int s = 0; s < 4; ++s) it.w[mt][s] = ldg16(wp + s * 512);
    }
    const int slot = lane & 15;
    const bool ok = slot < it.n;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const size_t o = (size_t)(it.p0 + slot) * kExpertWidth + s * kKStep + 8 * (lane >> 4);
        it.bh[s] = ok ? ldg16(P.h_hi + o) : z;
        it.bl[s] = ok ? ldg16(P.h_lo + o) : z;
    }
    it.tok = ok ? P.plan.toklist[it.tk + slot] : 0;
}

// acc[t][32 rows of the item's half] += the item's 32 x n block (the first
// tile of 16 tokens comes with the item; further tiles are loaded here).
template <int YS>
__device__ __forceinline__ void apply_down_item(const DNParams &P, const DownItem &it, int lane,
                                                float (*acc)[YS]) {
    const uint4 z = make_uint4(0, 0, 0, 0);
    for (int j = 0; j * 16 < it.n; ++j) {
        uint4 bh[4], bl[4];
        int t;
        const int slot = 16 * j + (lane & 15);
        const bool ok = slot < it.n;
        if (j == 0) {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                bh[s] = it.bh[s];
                bl[s] = it.bl[s];
            }
            t = it.tok;
        } else {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const size_t o =
                    (size_t)(it.p0 + slot) * kExpertWidth + s * kKStep + 8 * (lane >> 4);
                bh[s] = ok ? ldg16(P.h_hi + o) : z;
                bl[s] = ok ? ldg16(P.h_lo + o) : z;
            }
            t = ok ? P.plan.toklist[it.tk + slot] : 0;
        }
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
            f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                a = mfma16(it.w[mt][s], bh[s], a);
                a = mfma16(it.w[mt][s], bl[s], a);
            }
            if (ok) {
                float4 *dst = reinterpret_cast<float4 *>(
                    &acc[t][(2 * it.half + mt) * 16 + 4 * (lane >> 4)]);
                float4 v = *dst;
                v.x += a[0];
                v.y += a[1];
                v.z += a[2];
                v.w += a[3];
                *dst = v;
            }
        }
    }
}

template <int TB>
__global__ __launch_bounds__(256, 2) void down_dec_k(DNParams P) {
    constexpr int YS = kDnRows + 4;  // padded row stride of an accumulator
    __shared__ float yacc[4][TB][YS];
    __shared__ int s_flag;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int nU = P.plan.head[0];
    const int n_rb = P.d / kDnRows, RT = P.d / 16;
    // expert chunks: enough units for the resident workgroups, but at least
    // kDnMinPerChunk experts per chunk so each wavefront streams a pipeline
    int ES = (int)gridDim.x / n_rb;
    if (ES > nU / kDnMinPerChunk) ES = nU / kDnMinPerChunk;
    if (ES > kMaxChunks) ES = kMaxChunks;
    if (ES > 1 && (size_t)ES * P.T * P.d > P.ypart_elems) ES = (int)(P.ypart_elems / ((size_t)P.T * P.d));
    if (ES < 1) ES = 1;
    const int Uc = (nU + ES - 1) / ES;
    ES = (nU + Uc - 1) / Uc;
    const int units = n_rb * ES;
    float(*acc_w)[YS] = yacc[wv];

    for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int c = unit / n_rb, rb = unit - c * n_rb;
        for (int i = lane; i < P.T * YS; i += 64) acc_w[i / YS][i % YS] = 0.0f;
        // this wavefront's items: q -> (group c*Uc + wv + 4*(q/2), half q%2);
        // two items in flight, so the next item's loads overlap this one's math
        const int u0 = c * Uc + wv, u1 = min(nU, (c + 1) * Uc);
        const int nq = u0 < u1 ? 2 * ((u1 - u0 + 3) / 4) : 0;
        DownItem A, B;
        if (nq > 0) load_down_item(P, u0, 0, rb, RT, lane, A);
        for (int q = 0; q < nq; q += 2) {
            load_down_item(P, u0 + 4 * (q >> 1), 1, rb, RT, lane, B);
            apply_down_item<YS>(P, A, lane, acc_w);
            if (q + 2 < nq) load_down_item(P, u0 + 4 * ((q + 2) >> 1), 0, rb, RT, lane, A);
            apply_down_item<YS>(P, B, lane, acc_w);
        }
        __syncthreads();
        // sum the four accumulators in wavefront order
        for (int i = tid; i < P.T * (kDnRows / 4); i += blockDim.x) {
            const int t = i / (kDnRows / 4), r = 4 * (i - t * (kDnRows / 4));
            float4 s = *reinterpret_cast<const float4 *>(&yacc[0][t][r]);
#pragma unroll
            for (int w = 1; w < 4; ++w) {
                const float4 v = *reinterpret_cast<const float4 *>(&yacc[w][t][r]);
                s.x += v.x;
                s.y += v.y;
                s.z += v.z;
                s.w += v.w;
            }
            const size_t col = (size_t)rb * kDnRows + r;
            if (ES == 1) {
                *reinterpret_cast<float4 *>(P.y + (size_t)t * P.d + col) = s;
            } else {
                float *dst = P.ypart + ((size_t)c * P.T + t) * P.d + col;
                st_dev2(dst, s.x, s.y);
                st_dev2(dst + 2, s.z, s.w);
            }
        }
        if (ES > 1 && arrive_last(&P.cnt[rb], (unsigned)ES, &s_flag)) {
            // y[t][64 rows] = sum of the chunk partials in chunk order; every
            // thread owns up to kRedPer float2 of the block and issues the
            // loads of kRedChunks chunks at once
            constexpr int kRedPer = kDecodeTile * (kDnRows / 2) / 256;
            constexpr int kRedChunks = 4;
            const int nel = P.T * (kDnRows / 2);
            float2 acc[kRedPer];
            int off[kRedPer];
#pragma unroll
            for (int q = 0; q < kRedPer; ++q) {
                const int i = min(tid + 256 * q, nel - 1), t = i / (kDnRows / 2);
                off[q] = t * P.d + rb * kDnRows + 2 * (i - t * (kDnRows / 2));
                acc[q] = make_float2(0.f, 0.f);
            }
            const int nq = (nel - tid + 255) / 256;  // float2 owned by this thread
            for (int k0 = 0; k0 < ES; k0 += kRedChunks) {
                float2 v[kRedChunks][kRedPer];
#pragma unroll
                for (int k = 0; k < kRedChunks; ++k) {
                    const float *base = P.ypart + (size_t)min(k0 + k, ES - 1) * P.T * P.d;
#pragma unroll
                    for (int q = 0; q < kRedPer; ++q)
                        v[k][q] = q < nq ? ld_dev2(base + off[q]) : make_float2(0.f, 0.f);
                }
#pragma unroll
                for (int k = 0; k < kRedChunks; ++k)
                    if (k0 + k < ES)
#pragma unroll
                        for (int q = 0; q < kRedPer; ++q) {
                            acc[q].x += v[k][q].x;
                            acc[q].y += v[k][q].y;
                        }
            }
#pragma unroll
            for (int q = 0; q < kRedPer; ++q)
                if (q < nq) *reinterpret_cast<float2 *>(P.y + off[q]) = acc[q];
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ launchers

template <int TB>
void launch_down_dec_tb(const DNParams &P, int num_cu, hipStream_t s) {
    static const int occ = resident(down_dec_k<TB>, 256);
    hipLaunchKernelGGL(down_dec_k<TB>, dim3(occ * num_cu), dim3(256), 0, s, P);
}

}  // namespace

hipError_t launch_decode_ffn(pp_layer *L, const uint16_t *x, int T, float *y, hipStream_t s) {
    static const int occ = resident(gateup_dec_k, kGuThreads);
    const counter_layout cl = counters_for(L->dm, L->max_tokens);
    const GUParams gp = gu_params(L, x, T, false);
    prof_mark(L, PP_KERNEL_GATEUP, s, true);
    hipLaunchKernelGGL(gateup_dec_k, dim3(occ * L->num_cu), dim3(kGuThreads), 0, s, gp);
    prof_mark(L, PP_KERNEL_GATEUP, s, false);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    DNParams dp;
    dp.T = T;
    dp.d = L->dm.d;
    dp.E = L->dm.E;
    dp.Wd = L->Wd;
    dp.h_hi = L->h_hi;
    dp.h_lo = L->h_lo;
    dp.y = y;
    dp.ypart = L->ypart;
    dp.ypart_elems = L->ypart_elems;
    dp.cnt = L->counters + cl.down_base();
    dp.plan = plan_view(L, false);
    prof_mark(L, PP_KERNEL_DOWN, s, true);
    if (T <= 16)
        launch_down_dec_tb<16>(dp, L->num_cu, s);
    else if (T <= 32)
        launch_down_dec_tb<32>(dp, L->num_cu, s);
    else
        launch_down_dec_tb<64>(dp, L->num_cu, s);
    prof_mark(L, PP_KERNEL_DOWN, s, false);
    return hipGetLastError();
}

}  // namespace pp
