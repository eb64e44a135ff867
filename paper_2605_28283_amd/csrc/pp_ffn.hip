// Sparse expert evaluation: Eq. (ffn) restricted to the kept experts and
// summed per token, Eqs. (moefication_decomp) and (moe_output).
//
// Both paths work on "groups": one expert together with up to 64 of the tokens
// that kept it.  Decode (T <= 64) has one group per expert in the batch union;
// prefill splits each expert's token bucket into groups of 64.  Every (token,
// expert) pair gets a row in the h scratch; pairs are numbered expert by
// expert, tokens ascending inside an expert.
//
//   gateup_k  : per (group, K-slice) unit, 8 wavefronts = the expert's 8 tiles
//               of 16 neurons.  The group's token rows are staged in LDS in
//               MFMA B-operand order; the gate and up fragments stream from
//               HBM as contiguous 1 KiB wavefront loads (expert-major repack)
//               into bf16 MFMA 16x16x32 with fp32 accumulation.  With one
//               K-slice the epilogue forms h = SiLU(a) * b [* sigmoid(g_e)]
//               directly; with several, partial (a, b) rows are stored and the
//               last slice to arrive sums them in slice order.  h is stored as
//               a pair of bf16 numbers hi = bf16(h), lo = bf16(h - hi), so the
//               down projection keeps ~16 significant bits of h.
//   down_dec_k: decode down projection.  Unit = (row block of d, chunk of
//               union experts); accumulates y[rows, tokens] over the chunk with
//               two MFMAs per fragment (hi and lo); chunks are summed in a
//               fixed order by the last one to arrive.  No float atomics.
//   dispatch_k: prefill bucketing: per expert, the ascending list of tokens
//               that kept it (histogram + block scan + scatter), and y := 0.
//   down_pf_k : prefill down projection.  Unit = (group, row block); the
//               group's outputs are added into y with fp32 atomics.
#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kXBufBytes = 64 * 1024;

struct GUParams {
    const uint16_t *x;
    int T, d, E, NS;
    const uint16_t *Wgu;
    const uint32_t *selmask;
    const float *gsig;
    uint32_t flags;
    const int32_t *ecount;
    const int32_t *tokl;
    int tokl_stride;
    float *abpart;
    size_t abpart_rows;
    uint32_t *cnt;
    uint16_t *h_hi;
    uint16_t *h_lo;
};

struct DNParams {
    int T, d, E;
    const uint16_t *Wd;
    const uint32_t *selmask;
    const uint16_t *h_hi;
    const uint16_t *h_lo;
    float *y;
    float *ypart;
    size_t ypart_elems;
    uint32_t *cnt;
    const int32_t *ecount;
    const int32_t *tokl;
    int tokl_stride;
};

// Shared tables describing the groups of one call.
struct GroupTables {
    uint64_t mask[kMaxExperts];  // decode: tokens of union slot g
    int e[kMaxExperts];          // decode: expert of union slot g
    int off[kMaxExperts + 1];    // decode: pair offset of slot g; prefill: pair offset of expert
    int cb[kMaxExperts + 1];     // prefill: first group index of expert
    int cnt[kMaxExperts];        // prefill: bucket size of expert
    int scan[32];
    int nG, npairs, flag;
};

// Decode: groups = experts kept by at least one of the T <= 64 tokens.
__device__ void decode_groups(const uint32_t *__restrict__ selmask, int T, int E, GroupTables &G,
                              uint32_t (*sel)[8]) {
    const int tid = threadIdx.x;
    for (int i = tid; i < T * 8; i += blockDim.x) sel[i >> 3][i & 7] = selmask[i];
    __syncthreads();
    uint64_t m = 0;
    const int e = tid;
    if (e < E) {
        const int w = e >> 5, b = e & 31;
        for (int t = 0; t < T; ++t)
            if ((sel[t][w] >> b) & 1u) m |= 1ull << t;
    }
    const int act = (e < E && m != 0) ? 1 : 0;
    const int pc = (e < E) ? __popcll(m) : 0;
    int slot, poff, nU, npairs;
    block_excl_scan2(act, pc, &slot, &poff, &nU, &npairs, G.scan);
    if (act) {
        G.mask[slot] = m;
        G.e[slot] = e;
        G.off[slot] = poff;
    }
    if (tid == 0) {
        G.nG = nU;
        G.npairs = npairs;
    }
    __syncthreads();
}

// Prefill: groups = 64-token pieces of each expert's bucket.
__device__ void prefill_groups(const int32_t *__restrict__ ecount, int E, GroupTables &G) {
    const int tid = threadIdx.x;
    const int c = (tid < E) ? ecount[tid] : 0;
    const int nch = (c + kGroupTokens - 1) / kGroupTokens;
    int cb, off, nG, npairs;
    block_excl_scan2(nch, c, &cb, &off, &nG, &npairs, G.scan);
    if (tid < E) {
        G.cb[tid] = cb;
        G.off[tid] = off;
        G.cnt[tid] = c;
    }
    if (tid == 0) {
        G.cb[E] = nG;
        G.nG = nG;
        G.npairs = npairs;
    }
    __syncthreads();
}

// Expert owning prefill group g: largest e with cb[e] <= g (cb is non-decreasing).
__device__ __forceinline__ int group_expert(const GroupTables &G, int E, int g) {
    int lo = 0, hi = E - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (G.cb[mid] <= g)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Group g's expert, token count and first pair row; fills stok[0..n-1].
template <int MODE>
__device__ __forceinline__ void group_info(const GroupTables &G, int E, int g,
                                           const int32_t *__restrict__ tokl, int tokl_stride,
                                           int *e_out, int *n_out, int *poff_out, int *stok) {
    const int tid = threadIdx.x;
    if (MODE == 0) {
        const uint64_t m = G.mask[g];
        if (tid < 64 && ((m >> tid) & 1ull)) stok[__popcll(m & ((1ull << tid) - 1ull))] = tid;
        *e_out = G.e[g];
        *n_out = __popcll(m);
        *poff_out = G.off[g];
    } else {
        const int e = group_expert(G, E, g);
        const int c = g - G.cb[e];
        const int n = min(kGroupTokens, G.cnt[e] - c * kGroupTokens);
        if (tid < n) stok[tid] = tokl[(size_t)e * tokl_stride + c * kGroupTokens + tid];
        *e_out = e;
        *n_out = n;
        *poff_out = G.off[e] + c * kGroupTokens;
    }
}

__device__ __forceinline__ void store_h4(uint16_t *hi_row, uint16_t *lo_row, float h0, float h1,
                                         float h2, float h3) {
    const uint16_t a0 = f32_to_bf16(h0), a1 = f32_to_bf16(h1), a2 = f32_to_bf16(h2),
                   a3 = f32_to_bf16(h3);
    const uint16_t b0 = f32_to_bf16(h0 - bf16_to_f32(a0)), b1 = f32_to_bf16(h1 - bf16_to_f32(a1)),
                   b2 = f32_to_bf16(h2 - bf16_to_f32(a2)), b3 = f32_to_bf16(h3 - bf16_to_f32(a3));
    *reinterpret_cast<uint2 *>(hi_row) =
        make_uint2(a0 | ((uint32_t)a1 << 16), a2 | ((uint32_t)a3 << 16));
    *reinterpret_cast<uint2 *>(lo_row) =
        make_uint2(b0 | ((uint32_t)b1 << 16), b2 | ((uint32_t)b3 << 16));
}

template <int MODE>
__global__ __launch_bounds__(512) void gateup_k(GUParams P) {
    __shared__ uint4 xf[kXBufBytes / 16];
    __shared__ GroupTables G;
    __shared__ uint32_t sel[kDecodeTile][8];
    __shared__ int stok[kGroupTokens];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

    if (MODE == 0)
        decode_groups(P.selmask, P.T, P.E, G, sel);
    else
        prefill_groups(P.ecount, P.E, G);
    const int nG = G.nG, npairs = G.npairs;
    // K-slices per group: as many as keep every unit in the one round of
    // resident workgroups (gridDim.x), each slice at least kMinStepsPerSlice
    int KS = (int)gridDim.x / nG;
    const int max_ks = P.NS / kMinStepsPerSlice > 0 ? P.NS / kMinStepsPerSlice : 1;
    if (KS > max_ks) KS = max_ks;
    if (KS > 1 && (size_t)KS * npairs > P.abpart_rows) KS = (int)(P.abpart_rows / npairs);
    if (KS < 1) KS = 1;
    const int units = nG * KS;
    const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
    const uint4 z = make_uint4(0, 0, 0, 0);

    for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int g = unit / KS, ks = unit % KS;
        int e, n, poff;
        group_info<MODE>(G, P.E, g, P.tokl, P.tokl_stride, &e, &n, &poff, stok);
        __syncthreads();
        const int NT = (n + 15) >> 4;
        const int s0 = (int)((long)ks * P.NS / KS), s1 = (int)((long)(ks + 1) * P.NS / KS);
        const int nsc_max = kXBufBytes / (NT * 16 * 64);
        f32x4 ag[4], au[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            ag[j] = f32x4{0.f, 0.f, 0.f, 0.f};
            au[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        const uint16_t *wbase = P.Wgu + (size_t)(e * 8 + wv) * P.NS * 1024 + lane * 8;
        for (int sc = s0; sc < s1; sc += nsc_max) {
            const int nsc = min(nsc_max, s1 - sc);
            const int total = NT * 16 * nsc * 4;
            for (int c = tid; c < total; c += blockDim.x) {
                const int q = c / (nsc * 4), r = c - q * (nsc * 4);
                const int sl = r >> 2, qu = r & 3;
                uint4 v = z;
                if (q < n) v = ldg16(P.x + (size_t)stok[q] * P.d + (sc + sl) * kKStep + 8 * qu);
                xf[((q >> 4) * nsc + sl) * 64 + (q & 15) + 16 * qu] = v;
            }
            __syncthreads();
#pragma unroll 4
            for (int sl = 0; sl < nsc; ++sl) {
                const uint16_t *wp = wbase + (size_t)(sc + sl) * 1024;
                const uint4 wg = ldg16(wp);
                const uint4 wu = ldg16(wp + 512);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (j < NT) {
                        const uint4 b = xf[(j * nsc + sl) * 64 + lane];
                        ag[j] = mfma16(wg, b, ag[j]);
                        au[j] = mfma16(wu, b, au[j]);
                    }
                }
            }
            __syncthreads();
        }
        // lane holds neurons r0..r0+3 of token slot q = 16 j + lane%16
        const int r0 = wv * 16 + 4 * (lane >> 4);
        if (KS == 1) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int q = 16 * j + (lane & 15);
                if (j < NT && q < n) {
                    const float scl = sig ? P.gsig[(size_t)stok[q] * P.E + e] : 1.0f;
                    const size_t row = (size_t)(poff + q) * kExpertWidth + r0;
                    store_h4(P.h_hi + row, P.h_lo + row, silu(ag[j][0]) * au[j][0] * scl,
                             silu(ag[j][1]) * au[j][1] * scl, silu(ag[j][2]) * au[j][2] * scl,
                             silu(ag[j][3]) * au[j][3] * scl);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int q = 16 * j + (lane & 15);
                if (j < NT && q < n) {
                    float *row = P.abpart + ((size_t)ks * npairs + poff + q) * 256 + r0;
                    st_dev2(row, ag[j][0], ag[j][1]);
                    st_dev2(row + 2, ag[j][2], ag[j][3]);
                    st_dev2(row + 128, au[j][0], au[j][1]);
                    st_dev2(row + 130, au[j][2], au[j][3]);
                }
            }
            if (arrive_last(&P.cnt[g], (unsigned)KS, &G.flag)) {
                for (int i = tid; i < n * (kExpertWidth / 2); i += blockDim.x) {
                    const int q = i >> 6, r = 2 * (i & 63);
                    float2 a = make_float2(0.f, 0.f), b = make_float2(0.f, 0.f);
                    for (int k0 = 0; k0 < KS; k0 += 8) {
                        float2 u[8], v[8];
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            u[k] = v[k] = make_float2(0.f, 0.f);
                            if (k0 + k < KS) {
                                const float *row =
                                    P.abpart + ((size_t)(k0 + k) * npairs + poff + q) * 256;
                                u[k] = ld_dev2(row + r);
                                v[k] = ld_dev2(row + 128 + r);
                            }
                        }
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            a.x += u[k].x;
                            a.y += u[k].y;
                            b.x += v[k].x;
                            b.y += v[k].y;
                        }
                    }
                    const float scl = sig ? P.gsig[(size_t)stok[q] * P.E + e] : 1.0f;
                    const float h0 = silu(a.x) * b.x * scl, h1 = silu(a.y) * b.y * scl;
                    const uint16_t hi0 = f32_to_bf16(h0), hi1 = f32_to_bf16(h1);
                    const uint16_t lo0 = f32_to_bf16(h0 - bf16_to_f32(hi0)),
                                   lo1 = f32_to_bf16(h1 - bf16_to_f32(hi1));
                    const size_t o = (size_t)(poff + q) * kExpertWidth + r;
                    *reinterpret_cast<uint32_t *>(P.h_hi + o) = hi0 | ((uint32_t)hi1 << 16);
                    *reinterpret_cast<uint32_t *>(P.h_lo + o) = lo0 | ((uint32_t)lo1 << 16);
                }
            }
        }
        __syncthreads();
    }
}

template <int MT, int NTB>
__global__ __launch_bounds__(256) void down_dec_k(DNParams P) {
    __shared__ uint4 hfh[NTB * 4 * 64];
    __shared__ uint4 hfl[NTB * 4 * 64];
    __shared__ GroupTables G;
    __shared__ uint32_t sel[kDecodeTile][8];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    decode_groups(P.selmask, P.T, P.E, G, sel);
    const int nU = G.nG;
    const int RB = 64 * MT, n_rb = P.d / RB;
    int ES = (int)gridDim.x / n_rb;  // expert chunks: one round of resident workgroups
    if (ES > nU) ES = nU;
    if (ES > 1 && (size_t)ES * P.T * P.d > P.ypart_elems) ES = (int)(P.ypart_elems / ((size_t)P.T * P.d));
    if (ES < 1) ES = 1;
    const int Uc = (nU + ES - 1) / ES;
    ES = (nU + Uc - 1) / Uc;
    const int units = n_rb * ES;
    const int RT = P.d / 16;
    const uint4 z = make_uint4(0, 0, 0, 0);

    for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int rb = unit / ES, c = unit - rb * ES;
        f32x4 acc[MT][NTB];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int j = 0; j < NTB; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int u0 = c * Uc, u1 = min(nU, u0 + Uc);
        for (int u = u0; u < u1; ++u) {
            const int e = G.e[u];
            const uint64_t m = G.mask[u];
            const int poff = G.off[u];
            uint4 w[MT][4];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int rt = (rb * 4 + wv) * MT + mt;
                const uint16_t *wp = P.Wd + (((size_t)e * RT + rt) * 4 * 64 + lane) * 8;
#pragma unroll
                for (int s = 0; s < 4; ++s) w[mt][s] = ldg16(wp + s * 512);
            }
            __syncthreads();
            for (int i = tid; i < NTB * 4 * 64; i += blockDim.x) {
                const int j = i >> 8, s = (i >> 6) & 3, l = i & 63;
                const int t = 16 * j + (l & 15);
                uint4 hi = z, lo = z;
                if (t < P.T && ((m >> t) & 1ull)) {
                    const int p = poff + __popcll(m & ((1ull << t) - 1ull));
                    const size_t o = (size_t)p * kExpertWidth + s * kKStep + 8 * (l >> 4);
                    hi = ldg16(P.h_hi + o);
                    lo = ldg16(P.h_lo + o);
                }
                hfh[i] = hi;
                hfl[i] = lo;
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < NTB; ++j) {
                if ((m >> (16 * j)) & 0xFFFFull) {
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
        }
        // lane holds rows r0..r0+3 of token t = 16 j + lane%16
        if (ES == 1) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int r0 = ((rb * 4 + wv) * MT + mt) * 16 + 4 * (lane >> 4);
#pragma unroll
                for (int j = 0; j < NTB; ++j) {
                    const int t = 16 * j + (lane & 15);
                    if (t < P.T)
                        *reinterpret_cast<float4 *>(P.y + (size_t)t * P.d + r0) =
                            make_float4(acc[mt][j][0], acc[mt][j][1], acc[mt][j][2], acc[mt][j][3]);
                }
            }
        } else {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int r0 = ((rb * 4 + wv) * MT + mt) * 16 + 4 * (lane >> 4);
#pragma unroll
                for (int j = 0; j < NTB; ++j) {
                    const int t = 16 * j + (lane & 15);
                    if (t < P.T) {
                        float *row = P.ypart + ((size_t)c * P.T + t) * P.d + r0;
                        st_dev2(row, acc[mt][j][0], acc[mt][j][1]);
                        st_dev2(row + 2, acc[mt][j][2], acc[mt][j][3]);
                    }
                }
            }
            if (arrive_last(&P.cnt[rb], (unsigned)ES, &G.flag)) {
                for (int i = tid; i < P.T * (RB / 2); i += blockDim.x) {
                    const int t = i / (RB / 2);
                    const int r = rb * RB + 2 * (i - t * (RB / 2));
                    float2 s = make_float2(0.f, 0.f);
                    for (int k0 = 0; k0 < ES; k0 += 8) {
                        float2 v[8];
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            v[k] = (k0 + k < ES)
                                       ? ld_dev2(P.ypart + ((size_t)(k0 + k) * P.T + t) * P.d + r)
                                       : make_float2(0.f, 0.f);
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            s.x += v[k].x;
                            s.y += v[k].y;
                        }
                    }
                    *reinterpret_cast<float2 *>(P.y + (size_t)t * P.d + r) = s;
                }
            }
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void dispatch_k(const uint32_t *__restrict__ selmask, int T,
                                                  int E, int32_t *__restrict__ ecount,
                                                  int32_t *__restrict__ tokl, int stride,
                                                  float *__restrict__ y, size_t ny4) {
    __shared__ int scan[8];
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
    if (tid == 0) ecount[e] = base;
    float4 *y4 = reinterpret_cast<float4 *>(y);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + tid; i < ny4;
         i += (size_t)gridDim.x * blockDim.x)
        y4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

template <int MT>
__global__ __launch_bounds__(256) void down_pf_k(DNParams P) {
    __shared__ uint4 hfh[4 * 4 * 64];
    __shared__ uint4 hfl[4 * 4 * 64];
    __shared__ GroupTables G;
    __shared__ int stok[kGroupTokens];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    prefill_groups(P.ecount, P.E, G);
    const int nG = G.nG;
    const int RB = 64 * MT, n_rb = P.d / RB;
    const int units = nG * n_rb;
    const int RT = P.d / 16;
    const uint4 z = make_uint4(0, 0, 0, 0);

    for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
        const int g = unit / n_rb, rb = unit - g * n_rb;
        int e, n, poff;
        group_info<1>(G, P.E, g, P.tokl, P.tokl_stride, &e, &n, &poff, stok);
        uint4 w[MT][4];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int rt = (rb * 4 + wv) * MT + mt;
            const uint16_t *wp = P.Wd + (((size_t)e * RT + rt) * 4 * 64 + lane) * 8;
#pragma unroll
            for (int s = 0; s < 4; ++s) w[mt][s] = ldg16(wp + s * 512);
        }
        for (int i = tid; i < 4 * 4 * 64; i += blockDim.x) {
            const int j = i >> 8, s = (i >> 6) & 3, l = i & 63;
            const int q = 16 * j + (l & 15);
            uint4 hi = z, lo = z;
            if (q < n) {
                const size_t o = (size_t)(poff + q) * kExpertWidth + s * kKStep + 8 * (l >> 4);
                hi = ldg16(P.h_hi + o);
                lo = ldg16(P.h_lo + o);
            }
            hfh[i] = hi;
            hfl[i] = lo;
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

// Resident workgroups per CU of a kernel (0 if the query fails).
template <typename K>
int resident(K kernel, int threads) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess) n = 0;
    return n;
}

template <int MT, int NTB>
hipError_t launch_down_dec_v(const DNParams &P, int num_cu, hipStream_t s) {
    static const int occ = resident(down_dec_k<MT, NTB>, 256);
    const dim3 grid((occ > 0 ? occ : 1) * num_cu);
    hipLaunchKernelGGL((down_dec_k<MT, NTB>), grid, dim3(256), 0, s, P);
    return hipGetLastError();
}

template <int MT>
hipError_t launch_down_dec(const DNParams &P, int NTB, int num_cu, hipStream_t s) {
    switch (NTB) {
    case 1: return launch_down_dec_v<MT, 1>(P, num_cu, s);
    case 2: return launch_down_dec_v<MT, 2>(P, num_cu, s);
    case 3: return launch_down_dec_v<MT, 3>(P, num_cu, s);
    default: return launch_down_dec_v<MT, 4>(P, num_cu, s);
    }
}

GUParams gu_params(pp_layer *L, const uint16_t *x, int T) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    GUParams P;
    P.x = x;
    P.T = T;
    P.d = dm.d;
    P.E = dm.E;
    P.NS = dm.NS;
    P.Wgu = L->Wgu;
    P.selmask = L->selmask;
    P.gsig = L->gsig;
    P.flags = L->flags;
    P.ecount = L->ecount;
    P.tokl = L->tokl;
    P.tokl_stride = L->max_tokens;
    P.abpart = L->abpart;
    P.abpart_rows = kAbPartRows;
    P.cnt = L->counters + cl.route;
    P.h_hi = L->h_hi;
    P.h_lo = L->h_lo;
    return P;
}

DNParams dn_params(pp_layer *L, int T, float *y) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    DNParams P;
    P.T = T;
    P.d = dm.d;
    P.E = dm.E;
    P.Wd = L->Wd;
    P.selmask = L->selmask;
    P.h_hi = L->h_hi;
    P.h_lo = L->h_lo;
    P.y = y;
    P.ypart = L->ypart;
    P.ypart_elems = L->ypart_elems;
    P.cnt = L->counters + cl.route + cl.gateup;
    P.ecount = L->ecount;
    P.tokl = L->tokl;
    P.tokl_stride = L->max_tokens;
    return P;
}

int pick_mt(int d, int T) {
    int mt = T <= 16 ? 1 : (T <= 32 ? 2 : 4);
    while (mt > 1 && (d / 64) % mt != 0) mt >>= 1;
    return mt;
}

}  // namespace

counter_layout counters_for(const pp_dims &dm, int max_tokens) {
    counter_layout c;
    c.route = (size_t)(max_tokens + kRouteTile - 1) / kRouteTile;
    c.gateup = (size_t)(dm.E > kUnitTarget ? dm.E : kUnitTarget);
    c.down = (size_t)(dm.d / 64);
    c.total = c.route + c.gateup + c.down;
    return c;
}

hipError_t launch_decode_ffn(pp_layer *L, const uint16_t *x, int T, float *y, hipStream_t s) {
    const GUParams gp = gu_params(L, x, T);
    static const int occ_gu = resident(gateup_k<0>, 512);
    prof_mark(L, PP_KERNEL_GATEUP, s, true);
    hipLaunchKernelGGL(gateup_k<0>, dim3((occ_gu > 0 ? occ_gu : 1) * L->num_cu), dim3(512), 0, s,
                       gp);
    prof_mark(L, PP_KERNEL_GATEUP, s, false);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const DNParams dp = dn_params(L, T, y);
    const int NTB = (T + 15) / 16;
    const int mt = pick_mt(L->dm.d, T);
    prof_mark(L, PP_KERNEL_DOWN, s, true);
    if (mt == 1)
        err = launch_down_dec<1>(dp, NTB, L->num_cu, s);
    else if (mt == 2)
        err = launch_down_dec<2>(dp, NTB, L->num_cu, s);
    else
        err = launch_down_dec<4>(dp, NTB, L->num_cu, s);
    prof_mark(L, PP_KERNEL_DOWN, s, false);
    return err;
}

hipError_t launch_prefill_ffn(pp_layer *L, const uint16_t *x, int T, float *y, hipStream_t s) {
    const pp_dims &dm = L->dm;
    prof_mark(L, PP_KERNEL_DISPATCH, s, true);
    hipLaunchKernelGGL(dispatch_k, dim3(dm.E), dim3(256), 0, s, L->selmask, T, dm.E, L->ecount,
                       L->tokl, L->max_tokens, y, (size_t)T * dm.d / 4);
    prof_mark(L, PP_KERNEL_DISPATCH, s, false);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const GUParams gp = gu_params(L, x, T);
    static const int occ_gu = resident(gateup_k<1>, 512);
    prof_mark(L, PP_KERNEL_GATEUP, s, true);
    hipLaunchKernelGGL(gateup_k<1>, dim3((occ_gu > 0 ? occ_gu : 1) * L->num_cu), dim3(512), 0, s,
                       gp);
    prof_mark(L, PP_KERNEL_GATEUP, s, false);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    const DNParams dp = dn_params(L, T, y);
    const int mt = pick_mt(dm.d, 64);
    static const int occ4 = resident(down_pf_k<4>, 256), occ2 = resident(down_pf_k<2>, 256),
                     occ1 = resident(down_pf_k<1>, 256);
    const int occ = mt == 4 ? occ4 : (mt == 2 ? occ2 : occ1);
    const dim3 grid((occ > 0 ? occ : 1) * L->num_cu);
    prof_mark(L, PP_KERNEL_DOWN, s, true);
    if (mt == 4)
        hipLaunchKernelGGL((down_pf_k<4>), grid, dim3(256), 0, s, dp);
    else if (mt == 2)
        hipLaunchKernelGGL((down_pf_k<2>), grid, dim3(256), 0, s, dp);
    else
        hipLaunchKernelGGL((down_pf_k<1>), grid, dim3(256), 0, s, dp);
    prof_mark(L, PP_KERNEL_DOWN, s, false);
    return hipGetLastError();
}

}  // namespace pp
