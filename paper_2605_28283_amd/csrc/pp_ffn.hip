// Sparse expert evaluation: Eq. (ffn) restricted to the kept experts and
// summed per token, Eqs. (moefication_decomp) and (moe_output).
//
// Work is organised in "groups" listed by a plan: one expert with up to 64 of
// the tokens that kept it.  A decode batch (T <= 64) has one group per expert
// in the batch union (gateup_k derives that plan from the router's per-expert
// token masks and stores it for the down projection); prefill splits each
// expert's token bucket into groups of 64 (dispatch_k writes that plan).  Each
// (token, expert) pair owns one row of the h scratch; rows are numbered group
// by group, tokens ascending inside a group.
//
//   gateup_k  : unit = (group, K-slice); 8 wavefronts = the expert's 8 tiles
//               of 16 neurons.  The group's token rows are staged in LDS in
//               MFMA B-operand order; gate and up fragments stream from HBM as
//               contiguous 1 KiB wavefront loads (expert-major repack), double
//               buffered in registers, into bf16 MFMA 16x16x32 with fp32
//               accumulation.  With one K-slice the epilogue forms
//               h = SiLU(a) * b [* sigmoid(g_e)] directly; with several,
//               partial (a, b) rows are handed to the slice that arrives last,
//               which sums them in slice order.  h is stored as two bf16
//               numbers, hi = bf16(h) and lo = bf16(h - hi), so the down
//               projection keeps ~16 significant bits of h.
//   down_dec_k: decode down projection.  Unit = (64 rows of d, chunk of
//               groups); each wavefront takes every fourth group of the chunk,
//               multiplies its 64x128 down block with the group's compact token
//               tiles (two MFMAs per fragment: hi and lo) and adds the result
//               into its own LDS accumulator [tokens][64 rows] -- no
//               synchronisation inside the chunk; the next group's fragments
//               are loaded while the current one is multiplied.  The four accumulators are
//               summed in wavefront order; chunks are summed in chunk order by
//               the last to arrive.  No float atomics: decode is deterministic.
//   dispatch_k: prefill bucketing (per expert, the ascending list of tokens
//               that kept it: block scan + scatter), y := 0, and the prefill
//               plan, written by the last expert to finish.
//   down_pf_k : prefill down projection.  Unit = (group, 256 rows); the
//               group's h is staged in LDS once, its outputs are added into y
//               with fp32 atomics.
#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kXBufBytes = 64 * 1024;
constexpr int kGuThreads = 512;
constexpr int kPF = 2;          // K-steps per register buffer in gateup_k (two buffers)
constexpr int kDnRows = 64;     // rows of d per decode down unit
constexpr int kMaxChunks = 32;  // expert chunks of the decode down projection
constexpr int kDnMinPerChunk = 8;  // experts per chunk at least (two per wavefront)

struct GUParams {
    const uint16_t *x;
    int T, d, E, NS;
    const uint16_t *Wgu;
    const float *gsig;
    uint32_t flags;
    PlanView plan;
    const unsigned long long *emask;  // decode: tokens that kept each expert
    float *abpart;
    size_t abpart_rows;
    uint32_t *cnt;
    uint16_t *h_hi;
    uint16_t *h_lo;
};

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

__device__ __forceinline__ void split_bf16(float h, uint16_t &hi, uint16_t &lo) {
    hi = f32_to_bf16(h);
    lo = f32_to_bf16(h - bf16_to_f32(hi));
}

// ------------------------------------------------------------------ gate/up

// Stage token rows of a K sub-chunk into LDS in B-operand order:
// xf[(j * nsc + step) * 64 + lane] holds token slot 16 j + lane % 16,
// columns 32 (sc + step) + 8 (lane / 16) .. +7.  All loads are issued first.
template <int NT>
__device__ __forceinline__ void stage_x(const GUParams &P, const int *stok, int n, int sc, int nsc,
                                        uint4 *xf) {
    constexpr int kPerThread = kXBufBytes / 16 / kGuThreads;
    constexpr int kBatch = 4;  // loads in flight per thread (register budget)
    const int per_tok = nsc * 4;
    const int total = NT * 16 * per_tok;
    const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i0 = 0; i0 < kPerThread; i0 += kBatch) {
        if (threadIdx.x + kGuThreads * i0 >= total) break;
        uint4 v[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int c = threadIdx.x + kGuThreads * (i0 + i);
            v[i] = z;
            if (c < total) {
                const int q = c / per_tok, r = c - q * per_tok;
                if (q < n)
                    v[i] = ldg16(P.x + (size_t)stok[q] * P.d + (sc + (r >> 2)) * kKStep + 8 * (r & 3));
            }
        }
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int c = threadIdx.x + kGuThreads * (i0 + i);
            if (c < total) {
                const int q = c / per_tok, r = c - q * per_tok;
                xf[((q >> 4) * nsc + (r >> 2)) * 64 + (q & 15) + 16 * (r & 3)] = v[i];
            }
        }
    }
}

__device__ __forceinline__ void load_wgu(const uint16_t *wb, int step, int last, uint4 (&G)[kPF],
                                         uint4 (&U)[kPF]) {
#pragma unroll
    for (int i = 0; i < kPF; ++i) {
        const uint16_t *p = wb + (size_t)min(step + i, last) * 1024;
        G[i] = ldg16(p);
        U[i] = ldg16(p + 512);
    }
}

template <int NT>
__device__ __forceinline__ void mfma_wgu(const uint4 *xf, int nsc, int sl0, int nvalid,
                                         const uint4 (&G)[kPF], const uint4 (&U)[kPF],
                                         f32x4 (&ag)[NT], f32x4 (&au)[NT], int lane) {
#pragma unroll
    for (int i = 0; i < kPF; ++i) {
        if (i < nvalid) {
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const uint4 b = xf[(j * nsc + sl0 + i) * 64 + lane];
                ag[j] = mfma16(G[i], b, ag[j]);
                au[j] = mfma16(U[i], b, au[j]);
            }
        }
    }
}

template <int NT>
__device__ void gateup_unit(const GUParams &P, int e, int n, int p0, int g, int ks, int KS,
                            int npairs, const int *stok, uint4 *xf, int *flag) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int s0 = (int)((long)ks * P.NS / KS), s1 = (int)((long)(ks + 1) * P.NS / KS);
    constexpr int nsc_max = kXBufBytes / (NT * 16 * 64);
    f32x4 ag[NT], au[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        ag[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        au[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const uint16_t *wb = P.Wgu + (size_t)(e * 8 + wv) * P.NS * 1024 + lane * 8;
    for (int sc = s0; sc < s1; sc += nsc_max) {
        const int nsc = min(nsc_max, s1 - sc), last = sc + nsc - 1;
        uint4 G0[kPF], U0[kPF], G1[kPF], U1[kPF];
        load_wgu(wb, sc, last, G0, U0);  // weights do not wait for the token staging
        stage_x<NT>(P, stok, n, sc, nsc, xf);
        __syncthreads();
        for (int b = 0; b < nsc; b += 2 * kPF) {
            if (b + kPF < nsc) load_wgu(wb, sc + b + kPF, last, G1, U1);
            mfma_wgu<NT>(xf, nsc, b, min(kPF, nsc - b), G0, U0, ag, au, lane);
            if (b + 2 * kPF < nsc) load_wgu(wb, sc + b + 2 * kPF, last, G0, U0);
            if (b + kPF < nsc) mfma_wgu<NT>(xf, nsc, b + kPF, min(kPF, nsc - b - kPF), G1, U1, ag, au, lane);
        }
        __syncthreads();
    }
    // lane holds neurons r0..r0+3 of token slot q = 16 j + lane % 16
    const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
    const int r0 = wv * 16 + 4 * (lane >> 4);
    if (KS == 1) {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int q = 16 * j + (lane & 15);
            if (q < n) {
                const float scl = sig ? P.gsig[(size_t)stok[q] * P.E + e] : 1.0f;
                uint16_t hi[4], lo[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) split_bf16(silu(ag[j][i]) * au[j][i] * scl, hi[i], lo[i]);
                const size_t row = (size_t)(p0 + q) * kExpertWidth + r0;
                *reinterpret_cast<uint2 *>(P.h_hi + row) =
                    make_uint2(hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16));
                *reinterpret_cast<uint2 *>(P.h_lo + row) =
                    make_uint2(lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16));
            }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int q = 16 * j + (lane & 15);
        if (q < n) {
            float *row = P.abpart + ((size_t)ks * npairs + p0 + q) * 256 + r0;
            st_dev2(row, ag[j][0], ag[j][1]);
            st_dev2(row + 2, ag[j][2], ag[j][3]);
            st_dev2(row + 128, au[j][0], au[j][1]);
            st_dev2(row + 130, au[j][2], au[j][3]);
        }
    }
    if (!arrive_last(&P.cnt[g], (unsigned)KS, flag)) return;
    // (a, b) of the group's n x 128 block = sum of the slice partials in slice
    // order; a thread owns up to kRedPer float2 of it and issues the loads of
    // kRedSlices slices at once
    constexpr int kRedPer = 2;
    constexpr int kRedSlices = 4;
    const int nel = n * (kExpertWidth / 2);
    const size_t slice = (size_t)npairs * 256;
    for (int i0 = 0; i0 < nel; i0 += kRedPer * kGuThreads) {
        float2 a[kRedPer], b[kRedPer];
        int off[kRedPer];
        const int nq = (nel - i0 - tid + kGuThreads - 1) / kGuThreads;
#pragma unroll
        for (int q = 0; q < kRedPer; ++q) {
            const int i = min(i0 + tid + kGuThreads * q, nel - 1);
            off[q] = (p0 + (i >> 6)) * 256 + 2 * (i & 63);
            a[q] = b[q] = make_float2(0.f, 0.f);
        }
        for (int k0 = 0; k0 < KS; k0 += kRedSlices) {
            float2 u[kRedSlices][kRedPer], v[kRedSlices][kRedPer];
#pragma unroll
            for (int k = 0; k < kRedSlices; ++k) {
                const float *base = P.abpart + (size_t)min(k0 + k, KS - 1) * slice;
#pragma unroll
                for (int q = 0; q < kRedPer; ++q) {
                    u[k][q] = q < nq ? ld_dev2(base + off[q]) : make_float2(0.f, 0.f);
                    v[k][q] = q < nq ? ld_dev2(base + off[q] + 128) : make_float2(0.f, 0.f);
                }
            }
#pragma unroll
            for (int k = 0; k < kRedSlices; ++k)
                if (k0 + k < KS)
#pragma unroll
                    for (int q = 0; q < kRedPer; ++q) {
                        a[q].x += u[k][q].x;
                        a[q].y += u[k][q].y;
                        b[q].x += v[k][q].x;
                        b[q].y += v[k][q].y;
                    }
        }
#pragma unroll
        for (int q = 0; q < kRedPer; ++q) {
            if (q < nq) {
                const int i = i0 + tid + kGuThreads * q;
                const int qq = i >> 6, r = 2 * (i & 63);
                const float scl = sig ? P.gsig[(size_t)stok[qq] * P.E + e] : 1.0f;
                uint16_t h0, l0, h1, l1;
                split_bf16(silu(a[q].x) * b[q].x * scl, h0, l0);
                split_bf16(silu(a[q].y) * b[q].y * scl, h1, l1);
                const size_t o = (size_t)(p0 + qq) * kExpertWidth + r;
                *reinterpret_cast<uint32_t *>(P.h_hi + o) = h0 | ((uint32_t)h1 << 16);
                *reinterpret_cast<uint32_t *>(P.h_lo + o) = l0 | ((uint32_t)l1 << 16);
            }
        }
    }
}

// Decode plan, derived by every workgroup from the per-expert token masks:
// groups = experts kept by at least one token, ascending; group u owns pair
// rows [pair_u, pair_u + popcount(mask_u)), tokens ascending.  Workgroup 0
// also stores it for the down projection.
struct DecodePlan {
    unsigned long long mask[kMaxExperts];
    int e[kMaxExperts];
    int pair[kMaxExperts];
    int scan[2 * (kGuThreads / 64)];
    int nG, npairs;
};

__device__ void decode_plan(const GUParams &P, DecodePlan &D) {
    const int tid = threadIdx.x, e = tid;
    const unsigned long long m = (e < P.E) ? P.emask[e] : 0ull;
    const int act = m != 0ull ? 1 : 0, pc = __popcll(m);
    int slot, poff, nG, npairs;
    block_excl_scan2(act, pc, &slot, &poff, &nG, &npairs, D.scan);
    if (act) {
        D.mask[slot] = m;
        D.e[slot] = e;
        D.pair[slot] = poff;
        if (blockIdx.x == 0) {
            P.plan.grp_e[slot] = e;
            P.plan.grp_pair[slot] = poff;
            P.plan.grp_n[slot] = pc;
            P.plan.grp_tok[slot] = poff;
            int r = 0;
            for (unsigned long long mm = m; mm; mm &= mm - 1)
                P.plan.toklist[poff + r++] = __builtin_ctzll(mm);
        }
    }
    if (tid == 0) {
        D.nG = nG;
        D.npairs = npairs;
        if (blockIdx.x == 0) {
            P.plan.head[0] = nG;
            P.plan.head[1] = npairs;
        }
    }
    __syncthreads();
}

template <int MODE>
__global__ __launch_bounds__(kGuThreads, 4) void gateup_k(GUParams P) {
    __shared__ uint4 xf[kXBufBytes / 16];
    __shared__ int stok[kGroupTokens];
    __shared__ int s_flag;
    __shared__ DecodePlan D;
    const int tid = threadIdx.x;
    if (MODE == 0) decode_plan(P, D);
    const int nG = MODE == 0 ? D.nG : P.plan.head[0];
    const int npairs = MODE == 0 ? D.npairs : P.plan.head[1];
    // K-slices per group: as many as keep every unit in the one round of
    // resident workgroups (gridDim.x), each slice at least kMinStepsPerSlice
    int KS = (int)gridDim.x / nG;
    const int max_ks = P.NS / kMinStepsPerSlice > 0 ? P.NS / kMinStepsPerSlice : 1;
    if (KS > max_ks) KS = max_ks;
    if (KS > 1 && (size_t)KS * npairs > P.abpart_rows) KS = (int)(P.abpart_rows / npairs);
    if (KS < 1) KS = 1;
    const int units = nG * KS;
    for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int g = unit / KS, ks = unit - g * KS;
        int e, n, p0;
        if (MODE == 0) {
            const unsigned long long m = D.mask[g];
            e = D.e[g];
            n = __popcll(m);
            p0 = D.pair[g];
            if (tid < 64 && ((m >> tid) & 1ull)) stok[__popcll(m & ((1ull << tid) - 1ull))] = tid;
        } else {
            e = P.plan.grp_e[g];
            n = P.plan.grp_n[g];
            p0 = P.plan.grp_pair[g];
            if (tid < n) stok[tid] = P.plan.toklist[P.plan.grp_tok[g] + tid];
        }
        __syncthreads();
        switch ((n + 15) >> 4) {
        case 1: gateup_unit<1>(P, e, n, p0, g, ks, KS, npairs, stok, xf, &s_flag); break;
        case 2: gateup_unit<2>(P, e, n, p0, g, ks, KS, npairs, stok, xf, &s_flag); break;
        case 3: gateup_unit<3>(P, e, n, p0, g, ks, KS, npairs, stok, xf, &s_flag); break;
        default: gateup_unit<4>(P, e, n, p0, g, ks, KS, npairs, stok, xf, &s_flag); break;
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ down (decode)

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

// ------------------------------------------------------------------ prefill

__global__ __launch_bounds__(256) void dispatch_k(const uint32_t *__restrict__ selmask, int T,
                                                  int E, int32_t *__restrict__ ecount,
                                                  int32_t *__restrict__ tokl, int stride,
                                                  float *__restrict__ y, size_t ny4,
                                                  uint32_t *cnt, PlanView plan) {
    __shared__ int scan[8];
    __shared__ int s_flag;
    const int e = blockIdx.x, tid = threadIdx.x;
    const int w = e >> 5, b = e & 31;
    int base = 0;
    for (int t0 = 0; t0 < T; t0 += blockDim.x) {
        const int t = t0 + tid;
        const int f = (t < T && ((selmask[(size_t)t * 8 + w] >> b) & 1u)) ? 1 : 0;
        int ex, ex1, tot, tot1;
        block_excl_scan2(f, 0, &ex, &ex1, &tot, &tot1, scan);
        if (f) tokl[(size_t)e * stride + base + ex] = t;
        base += tot;
    }
    if (tid == 0) st_dev_u32(reinterpret_cast<uint32_t *>(ecount + e), (uint32_t)base);
    float4 *y4 = reinterpret_cast<float4 *>(y);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + tid; i < ny4;
         i += (size_t)gridDim.x * blockDim.x)
        y4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (!arrive_last(cnt, (unsigned)E, &s_flag)) return;
    // prefill plan: expert e's bucket becomes ceil(c_e / 64) groups
    const int c = (tid < E) ? (int)ld_dev_u32(reinterpret_cast<uint32_t *>(ecount + tid)) : 0;
    const int nch = (c + kGroupTokens - 1) / kGroupTokens;
    int cb, off, nG, npairs;
    block_excl_scan2(nch, c, &cb, &off, &nG, &npairs, scan);
    for (int ch = 0; ch < nch; ++ch) {
        const int g = cb + ch;
        plan.grp_e[g] = tid;
        plan.grp_pair[g] = off + ch * kGroupTokens;
        plan.grp_n[g] = min(kGroupTokens, c - ch * kGroupTokens);
        plan.grp_tok[g] = tid * stride + ch * kGroupTokens;
    }
    if (tid == 0) {
        plan.head[0] = nG;
        plan.head[1] = npairs;
    }
}

template <int MT>
__global__ __launch_bounds__(256) void down_pf_k(DNParams P) {
    __shared__ uint4 hfh[4 * 4 * 64];
    __shared__ uint4 hfl[4 * 4 * 64];
    __shared__ int stok[kGroupTokens];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int nG = P.plan.head[0];
    const int RB = 64 * MT, n_rb = P.d / RB;
    const int units = nG * n_rb;
    const int RT = P.d / 16;
    const uint4 z = make_uint4(0, 0, 0, 0);

    for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int g = unit / n_rb, rb = unit - g * n_rb;
        const int e = P.plan.grp_e[g], n = P.plan.grp_n[g], p0 = P.plan.grp_pair[g];
        const int tk = P.plan.grp_tok[g];
        if (tid < n) stok[tid] = P.plan.toklist[tk + tid];
        uint4 w[MT][4];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int rt = (rb * 4 + wv) * MT + mt;
            const uint16_t *wp = P.Wd + (((size_t)e * RT + rt) * 4 * 64 + lane) * 8;
#pragma unroll
            for (int s = 0; s < 4; ++s) w[mt][s] = ldg16(wp + s * 512);
        }
        {
            uint4 hv[4], lv[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int i = tid + 256 * k;
                const int j = i >> 8, s = (i >> 6) & 3, l = i & 63;
                const int q = 16 * j + (l & 15);
                hv[k] = lv[k] = z;
                if (q < n) {
                    const size_t o = (size_t)(p0 + q) * kExpertWidth + s * kKStep + 8 * (l >> 4);
                    hv[k] = ldg16(P.h_hi + o);
                    lv[k] = ldg16(P.h_lo + o);
                }
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                hfh[tid + 256 * k] = hv[k];
                hfl[tid + 256 * k] = lv[k];
            }
        }
        __syncthreads();
        const int NT = (n + 15) >> 4;
        f32x4 acc[MT][4];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (j < NT) {
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    const uint4 bh = hfh[(j * 4 + s) * 64 + lane];
                    const uint4 bl = hfl[(j * 4 + s) * 64 + lane];
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        acc[mt][j] = mfma16(w[mt][s], bh, acc[mt][j]);
                        acc[mt][j] = mfma16(w[mt][s], bl, acc[mt][j]);
                    }
                }
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int r0 = ((rb * 4 + wv) * MT + mt) * 16 + 4 * (lane >> 4);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int q = 16 * j + (lane & 15);
                if (j < NT && q < n) {
                    float *yr = P.y + (size_t)stok[q] * P.d + r0;
                    atomicAdd(yr + 0, acc[mt][j][0]);
                    atomicAdd(yr + 1, acc[mt][j][1]);
                    atomicAdd(yr + 2, acc[mt][j][2]);
                    atomicAdd(yr + 3, acc[mt][j][3]);
                }
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ launchers

// Resident workgroups per CU of a kernel (1 if the query fails).
template <typename K>
int resident(K kernel, int threads) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1)
        n = 1;
    return n;
}

GUParams gu_params(pp_layer *L, const uint16_t *x, int T, bool prefill) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    GUParams P;
    P.x = x;
    P.T = T;
    P.d = dm.d;
    P.E = dm.E;
    P.NS = dm.NS;
    P.Wgu = L->Wgu;
    P.gsig = L->gsig;
    P.flags = L->flags;
    P.plan = plan_view(L, prefill);
    P.emask = L->emask;
    P.abpart = L->abpart;
    P.abpart_rows = kAbPartRows;
    P.cnt = L->counters + cl.route;
    P.h_hi = L->h_hi;
    P.h_lo = L->h_lo;
    return P;
}

DNParams dn_params(pp_layer *L, int T, float *y, bool prefill) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    DNParams P;
    P.T = T;
    P.d = dm.d;
    P.E = dm.E;
    P.Wd = L->Wd;
    P.h_hi = L->h_hi;
    P.h_lo = L->h_lo;
    P.y = y;
    P.ypart = L->ypart;
    P.ypart_elems = L->ypart_elems;
    P.cnt = L->counters + cl.route + cl.gateup;
    P.plan = plan_view(L, prefill);
    return P;
}

hipError_t launch_gateup(pp_layer *L, const uint16_t *x, int T, bool prefill, hipStream_t s) {
    static const int occ0 = resident(gateup_k<0>, kGuThreads), occ1 = resident(gateup_k<1>, kGuThreads);
    const GUParams gp = gu_params(L, x, T, prefill);
    prof_mark(L, PP_KERNEL_GATEUP, s, true);
    if (prefill)
        hipLaunchKernelGGL(gateup_k<1>, dim3(occ1 * L->num_cu), dim3(kGuThreads), 0, s, gp);
    else
        hipLaunchKernelGGL(gateup_k<0>, dim3(occ0 * L->num_cu), dim3(kGuThreads), 0, s, gp);
    prof_mark(L, PP_KERNEL_GATEUP, s, false);
    return hipGetLastError();
}

template <int TB>
void launch_down_dec_tb(const DNParams &P, int num_cu, hipStream_t s) {
    static const int occ = resident(down_dec_k<TB>, 256);
    hipLaunchKernelGGL(down_dec_k<TB>, dim3(occ * num_cu), dim3(256), 0, s, P);
}

}  // namespace

counter_layout counters_for(const pp_dims &dm, int max_tokens) {
    counter_layout c;
    c.route = 0;
    c.gateup = (size_t)plan_max_groups(dm, max_tokens);
    c.down = (size_t)(dm.d / kDnRows);
    c.dispatch = 1;
    c.total = c.route + c.gateup + c.down + c.dispatch;
    return c;
}

hipError_t launch_decode_ffn(pp_layer *L, const uint16_t *x, int T, float *y, hipStream_t s) {
    hipError_t err = launch_gateup(L, x, T, false, s);
    if (err != hipSuccess) return err;
    const DNParams dp = dn_params(L, T, y, false);
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

hipError_t launch_prefill_ffn(pp_layer *L, const uint16_t *x, int T, float *y, hipStream_t s) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    prof_mark(L, PP_KERNEL_DISPATCH, s, true);
    hipLaunchKernelGGL(dispatch_k, dim3(dm.E), dim3(256), 0, s, L->selmask, T, dm.E, L->ecount,
                       L->tokl, L->max_tokens, y, (size_t)T * dm.d / 4,
                       L->counters + cl.route + cl.gateup + cl.down, plan_view(L, true));
    prof_mark(L, PP_KERNEL_DISPATCH, s, false);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    err = launch_gateup(L, x, T, true, s);
    if (err != hipSuccess) return err;
    const DNParams dp = dn_params(L, T, y, true);
    int mt = 4;
    while (mt > 1 && (dm.d / 64) % mt != 0) mt >>= 1;
    static const int occ4 = resident(down_pf_k<4>, 256), occ2 = resident(down_pf_k<2>, 256),
                     occ1 = resident(down_pf_k<1>, 256);
    prof_mark(L, PP_KERNEL_DOWN, s, true);
    if (mt == 4)
        hipLaunchKernelGGL((down_pf_k<4>), dim3(occ4 * L->num_cu), dim3(256), 0, s, dp);
    else if (mt == 2)
        hipLaunchKernelGGL((down_pf_k<2>), dim3(occ2 * L->num_cu), dim3(256), 0, s, dp);
    else
        hipLaunchKernelGGL((down_pf_k<1>), dim3(occ1 * L->num_cu), dim3(256), 0, s, dp);
    prof_mark(L, PP_KERNEL_DOWN, s, false);
    return hipGetLastError();
}

}  // namespace pp
