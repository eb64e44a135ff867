// Gate/up projections of one group (one expert with up to 64 of its tokens)
// over one K-slice, shared by the decode and prefill kernels: Eq. (ffn)'s
// x W_gate and x W_up for the kept expert, Eq. (moefication_decomp).  With
// GATED false the layer is the non-gated GELU MLP (one input projection with
// a per-neuron bias, h = GELU(x W_fc + b_fc)), which Sec. 2.1's decomposition
// covers as well.
//
// The group's token rows are staged in LDS in MFMA B-operand order; gate and
// up fragments stream from HBM as contiguous 1 KiB wavefront loads
// (expert-major repack), double buffered in registers, into bf16 MFMA
// 16x16x32 with fp32 accumulation.  With one K-slice the epilogue forms
// h = SiLU(a) * b [* sigmoid(g_e)] directly; with several, partial (a, b) rows
// are handed to the slice that arrives last, which sums them in slice order.
// h is stored as two bf16 numbers, hi = bf16(h) and lo = bf16(h - hi), so the
// down projection keeps ~16 significant bits of h.
#pragma once
#include "pp_select.h"

namespace pp {
namespace {

constexpr int kXBufBytes = 64 * 1024;
constexpr int kGuThreads = 512;
constexpr int kPF = 2;          // K-steps per register buffer (two buffers) with up to 4 token tiles

struct GUParams {
    const uint16_t *x;
    int T, d, E, NS;
    const uint16_t *Wgu;
    const float *bfc;   // non-gated layers: [E][128] input bias in expert order
    const float *gsig;
    uint32_t flags;
    PlanView plan;
    const unsigned long long *emask;  // decode: tokens that kept each expert
    float *abpart;
    size_t abpart_rows;
    uint32_t *cnt;
    uint16_t *h_hi;
    uint16_t *h_lo;
    // single-token decode: the kernel selects the token's experts itself from
    // the router's partial logits (rp), instead of reading the token masks
    int select_here;
    RouteParams rp;
};

__device__ __forceinline__ void split_bf16(float h, uint16_t &hi, uint16_t &lo) {
    hi = f32_to_bf16(h);
    lo = f32_to_bf16(h - bf16_to_f32(hi));
}

// ------------------------------------------------------------------ gate/up

// Stage token rows of a K sub-chunk into LDS in B-operand order:
// xf[(j * nsc + step) * 64 + lane] holds token slot 16 j + lane % 16,
// columns 32 (sc + step) + 8 (lane / 16) .. +7.  Loads go out in batches,
// every lane of a batch loading unconditionally from an element index clamped
// into the group (native vectors, so the zeroing selects stay in registers);
// the batch loop ends on a wavefront-uniform bound.  XB: loads per thread
// in a batch (0: chosen by NT for the register budget of the decode kernels).
template <int NT, int XB>
__device__ __forceinline__ void stage_x(const GUParams &P, const int *stok, int n, int sc, int nsc,
                                        uint4 *xf) {
    constexpr int kPerThread = kXBufBytes / 16 / kGuThreads;
    constexpr int kBatch = XB > 0 ? XB : (NT >= 4 ? 2 : 4);  // loads in flight per thread
    static_assert(kPerThread % kBatch == 0, "whole batches");
    const int per_tok = nsc * 4;
    const int total = NT * 16 * per_tok;
    const int wave0 = __builtin_amdgcn_readfirstlane(threadIdx.x & ~63);
#pragma unroll
    for (int i0 = 0; i0 < kPerThread; i0 += kBatch) {
        if (wave0 + kGuThreads * i0 >= total) break;
        u32x4_t v[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int c = min((int)threadIdx.x + kGuThreads * (i0 + i), total - 1);
            const int q = c / per_tok, r = c - q * per_tok;
            v[i] = *reinterpret_cast<const u32x4_t *>(P.x + (size_t)stok[min(q, n - 1)] * P.d +
                                                      (sc + (r >> 2)) * kKStep + 8 * (r & 3));
        }
        // A lane past the end stores the last element again, the value that
        // element's own thread stores, so the stores need no branch either.
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int c = min((int)threadIdx.x + kGuThreads * (i0 + i), total - 1);
            const int q = c / per_tok, r = c - q * per_tok;
            // The empty asm consumes the loaded value on every lane, so the
            // compiler cannot turn the zeroing select into a guarded load.
            asm volatile("" : "+v"(v[i]));
            const u32x4_t w = q < n ? v[i] : u32x4_t{0u, 0u, 0u, 0u};
            xf[((q >> 4) * nsc + (r >> 2)) * 64 + (q & 15) + 16 * (r & 3)] = make_uint4(w.x, w.y, w.z, w.w);
        }
    }
}

// bf16 elements of one wavefront's weight block per K-step: gate and up
// fragments (1024), or the single input projection of a non-gated layer (512).
template <bool GATED>
constexpr int kStepElems = GATED ? 1024 : 512;

template <bool GATED, int PF, bool STREAM>
__device__ __forceinline__ void load_wgu(const uint16_t *wb, int step, int last, uint4 (&G)[PF],
                                         uint4 (&U)[PF]) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
        const uint16_t *p = wb + (size_t)min(step + i, last) * kStepElems<GATED>;
        G[i] = ldw16_if<STREAM>(p);
        if (GATED) U[i] = ldw16_if<STREAM>(p + 512);
    }
}

template <int NT, bool GATED, int PF>
__device__ __forceinline__ void mfma_wgu(const uint4 *xf, int nsc, int sl0, int nvalid,
                                         const uint4 (&G)[PF], const uint4 (&U)[PF],
                                         f32x4 (&ag)[NT], f32x4 (&au)[NT], int lane) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
        if (i < nvalid) {
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const uint4 b = xf[(j * nsc + sl0 + i) * 64 + lane];
                ag[j] = mfma16(G[i], b, ag[j]);
                if (GATED) au[j] = mfma16(U[i], b, au[j]);
            }
        }
    }
}

// GPT-2's GELU, tanh form: 0.5 a (1 + tanh(sqrt(2/pi) (a + 0.044715 a^3))).
__device__ __forceinline__ float gelu_tanh(float a) {
    const float u = 0.7978845608028654f * (a + 0.044715f * a * a * a);
    return 0.5f * a * (1.0f + tanhf(u));
}

// h of neuron r (0..127 inside expert e) from the projections' sums.
template <bool GATED>
__device__ __forceinline__ float act(const GUParams &P, int e, int r, float a, float b) {
    if (GATED) return silu(a) * b;
    return gelu_tanh(a + P.bfc[e * kExpertWidth + r]);
}

// PF: K-steps per register buffer; two buffers alternate, so PF steps of
// weights are in flight while the other PF are multiplied.
template <int NT, bool GATED, int PF, int XB, bool STREAM>
__device__ __forceinline__ void gateup_unit(const GUParams &P, int e, int n, int p0, int g, int ks, int KS,
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
    const uint16_t *wb = P.Wgu + (size_t)(e * 8 + wv) * P.NS * kStepElems<GATED> + lane * 8;
    for (int sc = s0; sc < s1; sc += nsc_max) {
        const int nsc = min(nsc_max, s1 - sc), last = sc + nsc - 1;
        uint4 G0[PF], U0[PF], G1[PF], U1[PF];
        load_wgu<GATED, PF, STREAM>(wb, sc, last, G0, U0);  // weights do not wait for the token staging
        stage_x<NT, XB>(P, stok, n, sc, nsc, xf);
        __syncthreads();
        for (int b = 0; b < nsc; b += 2 * PF) {
            if (b + PF < nsc) load_wgu<GATED, PF, STREAM>(wb, sc + b + PF, last, G1, U1);
            mfma_wgu<NT, GATED, PF>(xf, nsc, b, min(PF, nsc - b), G0, U0, ag, au, lane);
            if (b + 2 * PF < nsc) load_wgu<GATED, PF, STREAM>(wb, sc + b + 2 * PF, last, G0, U0);
            if (b + PF < nsc)
                mfma_wgu<NT, GATED, PF>(xf, nsc, b + PF, min(PF, nsc - b - PF), G1, U1, ag, au,
                                        lane);
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
                for (int i = 0; i < 4; ++i)
                    split_bf16(act<GATED>(P, e, r0 + i, ag[j][i], au[j][i]) * scl, hi[i], lo[i]);
                const size_t row = (size_t)(p0 + q) * kExpertWidth + r0;
                *reinterpret_cast<uint2 *>(P.h_hi + row) =
                    make_uint2(hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16));
                *reinterpret_cast<uint2 *>(P.h_lo + row) =
                    make_uint2(lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16));
            }
        }
        return;
    }
    {
        // each lane's four neurons as one 16-byte store (the lanes of a token
        // slot fill 64 contiguous bytes of its row)
        const auto pr = buf_rsrc(P.abpart, (unsigned)(P.abpart_rows * 256 * sizeof(float)));
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int q = 16 * j + (lane & 15);
            if (q < n) {
                const unsigned o = (unsigned)(((size_t)ks * npairs + p0 + q) * 256 + r0) * 4u;
                st_dev16(pr, o, ag[j]);
                if (GATED) st_dev16(pr, o + 128 * 4u, au[j]);
            }
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
                    v[k][q] = (GATED && q < nq) ? ld_dev2(base + off[q] + 128)
                                                : make_float2(0.f, 0.f);
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
                split_bf16(act<GATED>(P, e, r, a[q].x, b[q].x) * scl, h0, l0);
                split_bf16(act<GATED>(P, e, r + 1, a[q].y, b[q].y) * scl, h1, l1);
                const size_t o = (size_t)(p0 + qq) * kExpertWidth + r;
                *reinterpret_cast<uint32_t *>(P.h_hi + o) = h0 | ((uint32_t)h1 << 16);
                *reinterpret_cast<uint32_t *>(P.h_lo + o) = l0 | ((uint32_t)l1 << 16);
            }
        }
    }
}

// Decode plan, derived by every workgroup from the per-expert token masks:
// groups = experts kept by at least one token, ascending; group u owns pair
// rows [pair_u, pair_u + popcount(mask_u)), tokens ascending.  With GLOBAL,
// workgroup 0 also stores it in the plan arrays.
struct DecodePlan {
    unsigned long long mask[kMaxExperts];
    int e[kMaxExperts];
    int pair[kMaxExperts];
    int scan[2 * (kGuThreads / 64)];
    int nG, npairs;
};

// m: this thread's expert's token mask (P.emask[threadIdx.x], 0 past E).
template <bool GLOBAL>
__device__ __forceinline__ void decode_plan(const GUParams &P, DecodePlan &D, unsigned long long m) {
    const int tid = threadIdx.x, e = tid;
    const int act = m != 0ull ? 1 : 0, pc = __popcll(m);
    int slot, poff, nG, npairs;
    block_excl_scan2(act, pc, &slot, &poff, &nG, &npairs, D.scan);
    if (act) {
        D.mask[slot] = m;
        D.e[slot] = e;
        D.pair[slot] = poff;
        if (GLOBAL && blockIdx.x == 0) {
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
        if (GLOBAL && blockIdx.x == 0) {
            P.plan.head[0] = nG;
            P.plan.head[1] = npairs;
        }
    }
    __syncthreads();
}

// One group's gate/up unit, dispatched on its number of 16-token tiles (at
// most NTMAX: a kernel whose groups are known to be small is compiled without
// the larger tiles' registers and spends them on a deeper weight prefetch PF).
template <bool GATED, int NTMAX, int PF, bool STREAM, int XB = 0>
__device__ __forceinline__ void gateup_group(const GUParams &P, int e, int n, int p0, int g,
                                             int ks, int KS, int npairs, const int *stok,
                                             uint4 *xf, int *flag) {
    const int nt = (n + 15) >> 4;
    if (NTMAX >= 4 && nt >= 4)
        gateup_unit<(NTMAX >= 4 ? 4 : 1), GATED, PF, XB, STREAM>(P, e, n, p0, g, ks, KS, npairs, stok, xf, flag);
    else if (NTMAX >= 3 && nt == 3)
        gateup_unit<(NTMAX >= 3 ? 3 : 1), GATED, PF, XB, STREAM>(P, e, n, p0, g, ks, KS, npairs, stok, xf, flag);
    else if (NTMAX >= 2 && nt == 2)
        gateup_unit<(NTMAX >= 2 ? 2 : 1), GATED, PF, XB, STREAM>(P, e, n, p0, g, ks, KS, npairs, stok, xf, flag);
    else
        gateup_unit<1, GATED, PF, XB, STREAM>(P, e, n, p0, g, ks, KS, npairs, stok, xf, flag);
}

// Most K-slices a group is split into: each slice covers at least
// kMinStepsPerSlice K-steps, and a small union (at most kSmallUnion kept
// experts) takes at most kMaxSlicesSmallUnion slices per group: there the
// hand-off of more, shorter slices costs more than their streaming gains
// (d = 4096: T = 1, tau 0.9 and T = 8, tau 0.5 / 0.7 gain 1.2-1.8 us per
// step with 8 slices of 16 K-steps instead of 16 of 8).
__device__ __forceinline__ int max_slices(const GUParams &P, int nG) {
    int m = P.NS / kMinStepsPerSlice > 0 ? P.NS / kMinStepsPerSlice : 1;
    if (nG <= kSmallUnion && m > kMaxSlicesSmallUnion) m = kMaxSlicesSmallUnion;
    return m;
}

// K-slices per group: as many as keep all nG * KS units within `slots`
// workgroups, at most max_slices, and the partial rows within the abpart
// scratch.
__device__ __forceinline__ int choose_ks(const GUParams &P, int nG, int npairs, int slots) {
    int KS = nG > 0 ? slots / nG : 1;
    const int max_ks = max_slices(P, nG);
    if (KS > max_ks) KS = max_ks;
    if (KS > 1 && (size_t)KS * npairs > P.abpart_rows) KS = (int)(P.abpart_rows / npairs);
    return KS < 1 ? 1 : KS;
}

// Resident workgroups per CU of a kernel (1 if the query fails).
template <typename K>
int resident(K kernel, int threads) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1)
        n = 1;
    return n;
}

inline GUParams gu_params(pp_layer *L, const uint16_t *x, int T, bool prefill) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    GUParams P;
    P.x = x;
    P.T = T;
    P.d = dm.d;
    P.E = dm.E;
    P.NS = dm.NS;
    P.Wgu = L->Wgu;
    P.bfc = L->bfc;
    P.gsig = L->gsig;
    P.flags = L->flags;
    P.plan = plan_view(L, prefill);
    P.emask = L->emask;
    P.abpart = L->abpart;
    P.abpart_rows = kAbPartRows;
    P.cnt = L->counters + cl.gateup_base();
    P.h_hi = L->h_hi;
    P.h_lo = L->h_lo;
    P.select_here = 0;
    return P;
}

}  // namespace
}  // namespace pp
