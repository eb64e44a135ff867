// Prefill expert evaluation: Eq. (ffn) restricted to the kept experts and
// summed per token, Eqs. (moefication_decomp) and (moe_output), for large T.
//
// Work is organised in "groups" listed by a plan: one expert with up to 64 of
// the tokens that kept it.  dispatch_k buckets the tokens per expert and
// splits each bucket into groups of 64; each (token, expert) pair owns one
// row of the h scratch, rows numbered group by group, tokens ascending inside
// a group.
//
//   dispatch_k  : per expert, the ascending list of tokens that kept it (block
//                 scan + scatter) and the plan, written by the last expert to
//                 finish; when the batch has more pairs than the pair-row
//                 buffer holds, further workgroups set y to the output bias
//                 (0 for SwiGLU layers) for the atomic adds of the pairs past
//                 it.
//   gateup_pf_k : unit = (group, K-slice); the gate/up projections and the
//                 SiLU product of one group (shared with the decode kernel).
//   down_pf_k   : unit = (expert, 256 rows); the expert's down block stays in
//                 registers across its token groups; each (token, expert)
//                 pair's rows go to a pair-row buffer (pairs past its 1 GiB
//                 capacity add into y with fp32 atomics).
//   combine_pf_k: y[t] = output bias + t's pair rows, kept experts in
//                 ascending order (y[t] + the rows for a token with pairs past
//                 the buffer) -- no float atomics while the buffer holds every
//                 pair, so the result is deterministic.
// Units of one expert are placed on one XCD (shared weights or h in L2).
#include "pp_gateup.h"

namespace pp {
namespace {

struct DNParams {
    int T, d, E;
    const uint16_t *Wd;
    const uint16_t *h_hi;
    const uint16_t *h_lo;
    float *y;
    float *part;     // [cap][d] pair rows
    size_t cap;
    PlanView plan;
};

template <bool GATED>
__global__ __launch_bounds__(kGuThreads, 4) void gateup_pf_k(GUParams P) {
    __shared__ uint4 xf[kXBufBytes / 16];
    __shared__ int stok[kGroupTokens];
    __shared__ int s_flag;
    const int tid = threadIdx.x;
    const int nG = P.plan.head[0];
    const int npairs = P.plan.head[1];
    const int KS = choose_ks(P, nG, npairs, (int)gridDim.x);
    const int units = nG * KS;
    // consecutive units (K-slices of a group, then the groups of one expert)
    // go to the same XCD, where they share the expert's weights in L2
    const int slots = 8 * ((units + 7) / 8);
    for (int slot = blockIdx.x; slot < slots; slot += gridDim.x) {
        const int unit = xcd_order(slot, units);
        if (unit >= units) continue;
        const int g = unit / KS, ks = unit - g * KS;
        const int e = P.plan.grp_e[g];
        const int n = P.plan.grp_n[g];
        const int p0 = P.plan.grp_pair[g];
        if (tid < n) stok[tid] = P.plan.toklist[P.plan.grp_tok[g] + tid];
        __syncthreads();
        gateup_group<GATED, 4, kPF>(P, e, n, p0, g, ks, KS, npairs, stok, xf, &s_flag);
        __syncthreads();
    }
}

// ------------------------------------------------------------------ prefill

__global__ __launch_bounds__(256) void dispatch_k(const uint32_t *__restrict__ selmask,
                                                  const int32_t *__restrict__ count, size_t cap,
                                                  int T, int E, int32_t *__restrict__ ecount,
                                                  int32_t *__restrict__ tokl, int stride,
                                                  float *__restrict__ y, size_t ny4,
                                                  const float *__restrict__ bproj, int d4,
                                                  int32_t *__restrict__ posq,
                                                  int32_t *__restrict__ ebase, uint32_t *cnt,
                                                  PlanView plan) {
    __shared__ int scan[8];
    __shared__ int s_flag;
    const int e = blockIdx.x, tid = threadIdx.x;
    if (e >= E) {
        // workgroups past the experts set y to the output bias (or 0) if some
        // pairs will not fit the pair-row buffer and add into y instead
        static_assert(sizeof(scan) >= 4 * sizeof(int), "four wavefront sums");
        size_t c = 0;
        for (int t = tid; t < T; t += blockDim.x) c += (size_t)count[t];
        const int cw = __builtin_amdgcn_readlane(wave_scan_i32((int)c), 63);
        if ((tid & 63) == 0) scan[tid >> 6] = cw;
        __syncthreads();
        if ((size_t)scan[0] + scan[1] + scan[2] + scan[3] <= cap) return;
        float4 *y4 = reinterpret_cast<float4 *>(y);
        const float4 *b4 = reinterpret_cast<const float4 *>(bproj);
        const size_t nz = (size_t)(gridDim.x - E) * blockDim.x;
        for (size_t i = (size_t)(e - E) * blockDim.x + tid; i < ny4; i += nz)
            y4[i] = b4 ? b4[i % d4] : make_float4(0.f, 0.f, 0.f, 0.f);
        return;
    }
    const int w = e >> 5, b = e & 31;
    int base = 0;
    for (int t0 = 0; t0 < T; t0 += blockDim.x) {
        const int t = t0 + tid;
        const int f = (t < T && ((selmask[(size_t)t * 8 + w] >> b) & 1u)) ? 1 : 0;
        int ex, ex1, tot, tot1;
        block_excl_scan2(f, 0, &ex, &ex1, &tot, &tot1, scan);
        if (f) {
            tokl[(size_t)e * stride + base + ex] = t;
            posq[(size_t)t * E + e] = base + ex;
        }
        base += tot;
    }
    if (tid == 0) st_dev_u32(reinterpret_cast<uint32_t *>(ecount + e), (uint32_t)base);
    if (!arrive_last(cnt, (unsigned)E, &s_flag)) return;
    // prefill plan: expert e's bucket becomes ceil(c_e / 64) groups
    const int c = (tid < E) ? (int)ld_dev_u32(reinterpret_cast<uint32_t *>(ecount + tid)) : 0;
    const int nch = (c + kGroupTokens - 1) / kGroupTokens;
    int cb, off, nG, npairs;
    block_excl_scan2(nch, c, &cb, &off, &nG, &npairs, scan);
    if (tid < E) {
        plan.egrp[tid] = cb;
        ebase[tid] = off;
    }
    if (tid == 0) plan.egrp[E] = nG;
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

// Unit = (expert, 256 rows of d): the four wavefronts hold the expert's
// 256 x 128 down block in registers (four 16-row tiles each, loaded once) and
// run it over the expert's token groups of 64.  A group's h (hi and lo, MFMA B
// order) is staged in LDS while the next group's is being loaded; the
// 64 x 256 result is transposed through LDS and stored as the pairs' rows
// (each store instruction 64 consecutive floats of one pair's row), which
// combine_pf_k sums per token.  Pairs past the buffer's capacity add into y
// with fp32 atomics instead.  Units of one expert share its h rows and go to
// the same XCD.
constexpr int kPfRows = 256;
__global__ __launch_bounds__(256, 2) void down_pf_k(DNParams P) {
    constexpr int MT = 4;
    __shared__ union {
        struct {
            uint4 hi[4 * 4 * 64];  // [token tile][K-step][lane]
            uint4 lo[4 * 4 * 64];
        } h;
        float y[kGroupTokens][kPfRows];
    } S;
    __shared__ int stok[kGroupTokens];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int n_rb = (P.d + kPfRows - 1) / kPfRows;
    const int units = P.E * n_rb;
    const int slots = 8 * ((units + 7) / 8);
    const int RT = P.d / 16;
    const uint4 z = make_uint4(0, 0, 0, 0);

    for (int slot = blockIdx.x; slot < slots; slot += gridDim.x) {
        const int unit = xcd_order(slot, units);
        if (unit >= units) continue;
        const int e = unit / n_rb, rb = unit - e * n_rb;
        const int g0 = P.plan.egrp[e], g1 = P.plan.egrp[e + 1];
        if (g0 >= g1) continue;
        const int nrows = min(kPfRows, P.d - rb * kPfRows);
        uint4 w[MT][4];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int rt = min(rb * (kPfRows / 16) + wv * MT + mt, RT - 1);  // past d: unused
            const uint16_t *wp = P.Wd + (((size_t)e * RT + rt) * 4 * 64 + lane) * 8;
#pragma unroll
            for (int s = 0; s < 4; ++s) w[mt][s] = ldg16(wp + s * 512);
        }
        // h of one group in B-fragment order: thread slot i = tid + 256 k holds
        // token tile i / 256, K-step (i / 64) % 4, lane i % 64
        uint4 hv[4], lv[4];
        auto load_h = [&](int g) {
            const int n = P.plan.grp_n[g], p0 = P.plan.grp_pair[g];
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
        };
        load_h(g0);
        for (int g = g0; g < g1; ++g) {
            const int n = P.plan.grp_n[g];
            __syncthreads();  // the previous group's atomics have read S.y
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                S.h.hi[tid + 256 * k] = hv[k];
                S.h.lo[tid + 256 * k] = lv[k];
            }
            if (tid < n) stok[tid] = P.plan.toklist[P.plan.grp_tok[g] + tid];
            __syncthreads();
            if (g + 1 < g1) load_h(g + 1);
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
                        const uint4 bh = S.h.hi[(j * 4 + s) * 64 + lane];
                        const uint4 bl = S.h.lo[(j * 4 + s) * 64 + lane];
#pragma unroll
                        for (int mt = 0; mt < MT; ++mt) {
                            acc[mt][j] = mfma16(w[mt][s], bh, acc[mt][j]);
                            acc[mt][j] = mfma16(w[mt][s], bl, acc[mt][j]);
                        }
                    }
                }
            }
            __syncthreads();  // h is no longer read: its LDS becomes the transpose buffer
            // lane holds rows 4 (lane / 16) + i of its tile, token slot 16 j + lane % 16
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int r0 = (wv * MT + mt) * 16 + 4 * (lane >> 4);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (j < NT)
                        *reinterpret_cast<float4 *>(&S.y[16 * j + (lane & 15)][r0]) = make_float4(
                            acc[mt][j][0], acc[mt][j][1], acc[mt][j][2], acc[mt][j][3]);
            }
            __syncthreads();
            const int p0 = P.plan.grp_pair[g];
            for (int q = wv; q < n; q += 4) {
                const size_t pair = (size_t)(p0 + q);
                if (pair < P.cap) {  // the pair's row, summed per token by combine_pf_k
                    static_assert(kPfRows == 4 * 64, "one float4 per lane covers a row");
                    float4 *pr = reinterpret_cast<float4 *>(P.part + pair * P.d + (size_t)rb * kPfRows);
                    if (4 * lane < nrows) pr[lane] = *reinterpret_cast<const float4 *>(&S.y[q][4 * lane]);
                } else {  // past the buffer: straight into y
                    float *yr = P.y + (size_t)stok[q] * P.d + (size_t)rb * kPfRows;
#pragma unroll
                    for (int c = 0; c < kPfRows / 64; ++c)
                        if (64 * c + lane < nrows) atomicAdd(yr + 64 * c + lane, S.y[q][64 * c + lane]);
                }
            }
        }
    }
}

// y[t] = the output bias (or 0) + the rows of t's pairs, kept experts in
// ascending order (a fixed order: deterministic).  One workgroup per token:
// wavefront 0 lists the token's pair rows in LDS (a ballot prefix over the
// expert bitmask), then every thread sums its four float4 columns, eight rows
// at a time with all of a batch's loads in flight.  A token with pairs past
// the buffer starts from y instead, which then holds the output bias and
// those pairs' atomic contributions.
__global__ __launch_bounds__(256) void combine_pf_k(const uint32_t *__restrict__ selmask, int T,
                                                    int E, int d, const int32_t *__restrict__ posq,
                                                    const int32_t *__restrict__ ebase,
                                                    const float *__restrict__ part, size_t cap,
                                                    const float *__restrict__ bproj,
                                                    float *__restrict__ y) {
    constexpr int kBatch = 8;   // pair rows in flight
    constexpr int kChunks = 4;  // float4 columns per thread and row (d = 4096 in one pass)
    __shared__ int plist[kMaxExperts];
    __shared__ int s_k, s_spill;
    const int tid = threadIdx.x, lane = tid & 63;
    const int t = blockIdx.x;
    if (tid < 64) {
        const uint32_t *sm = selmask + (size_t)t * 8;
        int k = 0;
        bool spill = false;
        for (int e0 = 0; e0 < E; e0 += 64) {
            const int e = e0 + lane;
            const bool kept = e < E && ((sm[e >> 5] >> (e & 31)) & 1u);
            const unsigned long long bal = __ballot(kept);
            if (kept) {
                const size_t pair = (size_t)ebase[e] + posq[(size_t)t * E + e];
                plist[k + __popcll(bal & ((1ull << lane) - 1ull))] = pair < cap ? (int)pair : -1;
                spill = spill || pair >= cap;
            }
            k += __popcll(bal);
        }
        spill = __ballot(spill) != 0ull;
        if (lane == 0) {
            s_k = k;
            s_spill = spill ? 1 : 0;
        }
    }
    __syncthreads();
    const int k = s_k, d4 = d / 4;
    float4 *yt = reinterpret_cast<float4 *>(y + (size_t)t * d);
    // the starting value: y (bias + atomic adds) or the bias itself
    const float4 *y0 = s_spill ? yt : reinterpret_cast<const float4 *>(bproj);
    // a thread's kChunks float4 columns of kBatch rows are all in flight at once
    for (int c0 = 0; c0 < d4; c0 += kChunks * 256) {
        float4 acc[kChunks];
#pragma unroll
        for (int u = 0; u < kChunks; ++u) {
            const int c4 = c0 + tid + 256 * u;
            acc[u] = (c4 < d4 && y0) ? y0[c4] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        for (int i0 = 0; i0 < k; i0 += kBatch) {
            float4 v[kBatch][kChunks];
#pragma unroll
            for (int r = 0; r < kBatch; ++r) {
                const float4 *row =
                    reinterpret_cast<const float4 *>(part + (size_t)max(plist[min(i0 + r, k - 1)], 0) * d);
#pragma unroll
                for (int u = 0; u < kChunks; ++u) v[r][u] = row[min(c0 + tid + 256 * u, d4 - 1)];
            }
#pragma unroll
            for (int r = 0; r < kBatch; ++r) {
                if (i0 + r < k && plist[i0 + r] >= 0) {
#pragma unroll
                    for (int u = 0; u < kChunks; ++u) {
                        acc[u].x += v[r][u].x;
                        acc[u].y += v[r][u].y;
                        acc[u].z += v[r][u].z;
                        acc[u].w += v[r][u].w;
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kChunks; ++u) {
            const int c4 = c0 + tid + 256 * u;
            if (c4 < d4) yt[c4] = acc[u];
        }
    }
}

// ------------------------------------------------------------------ launchers

DNParams dn_params(pp_layer *L, int T, float *y) {
    DNParams P;
    P.T = T;
    P.d = L->dm.d;
    P.E = L->dm.E;
    P.Wd = L->Wd;
    P.h_hi = L->h_hi;
    P.h_lo = L->h_lo;
    P.y = y;
    P.part = L->pf_part;
    P.cap = L->pf_cap;
    P.plan = plan_view(L, true);
    return P;
}

}  // namespace

counter_layout counters_for(const pp_dims &dm, int max_tokens) {
    counter_layout c;
    c.route = 0;
    c.gateup = (size_t)plan_max_groups(dm, max_tokens);
    c.down = (size_t)((dm.d + 127) / 128);
    c.dispatch = 1;
    c.total = c.route + c.gateup + c.down + c.dispatch;
    return c;
}

hipError_t launch_prefill_ffn(pp_layer *L, const uint16_t *x, int T, const int32_t *count,
                              float *y, hipStream_t s) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    prof_mark(L, PP_KERNEL_DISPATCH, s, true);
    hipLaunchKernelGGL(dispatch_k, dim3(dm.E + L->num_cu), dim3(256), 0, s, L->selmask, count,
                       L->pf_cap, T, dm.E, L->ecount,
                       L->tokl, L->max_tokens, y, (size_t)T * dm.d / 4, L->bproj, dm.d / 4,
                       L->pf_posq, L->pf_ebase, L->counters + cl.dispatch_base(),
                       plan_view(L, true));
    prof_mark(L, PP_KERNEL_DISPATCH, s, false);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    static const int occ_g = resident(gateup_pf_k<true>, kGuThreads);
    static const int occ_p = resident(gateup_pf_k<false>, kGuThreads);
    const GUParams gp = gu_params(L, x, T, true);
    prof_mark(L, PP_KERNEL_GATEUP, s, true);
    if (L->gated)
        hipLaunchKernelGGL(gateup_pf_k<true>, dim3(occ_g * L->num_cu), dim3(kGuThreads), 0, s, gp);
    else
        hipLaunchKernelGGL(gateup_pf_k<false>, dim3(occ_p * L->num_cu), dim3(kGuThreads), 0, s, gp);
    prof_mark(L, PP_KERNEL_GATEUP, s, false);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    const DNParams dp = dn_params(L, T, y);
    static const int occ_dn = resident(down_pf_k, 256);
    prof_mark(L, PP_KERNEL_DOWN, s, true);
    hipLaunchKernelGGL(down_pf_k, dim3(occ_dn * L->num_cu), dim3(256), 0, s, dp);
    hipLaunchKernelGGL(combine_pf_k, dim3(T), dim3(256), 0, s, L->selmask, T, dm.E, dm.d,
                       L->pf_posq, L->pf_ebase, L->pf_part, L->pf_cap, L->bproj, y);
    prof_mark(L, PP_KERNEL_DOWN, s, false);
    return hipGetLastError();
}

}  // namespace pp
