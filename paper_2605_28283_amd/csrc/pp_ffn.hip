// Prefill expert evaluation: Eq. (ffn) restricted to the kept experts and
// summed per token, Eqs. (moefication_decomp) and (moe_output), for large T.
//
// Work is organised in "groups" listed by a plan: one expert with up to 128
// of the tokens that kept it.  dispatch_k buckets the tokens per expert and
// splits each bucket into groups of 128; each (token, expert) pair owns one
// row of the h scratch, rows numbered group by group, tokens ascending inside
// a group.
//
//   dispatch_k  : per expert, the ascending list of tokens that kept it
//                 (ballot prefix over blocks of 256 tokens + scatter), where
//                 each chunk of kPfChunk tokens starts in it, and the plan,
//                 written by the last expert to finish.
//   gateup_pf_k : unit = one group, all of K, one workgroup per CU; the
//                 gate/up projections and the SiLU product (bf16 MFMA, each
//                 weight fragment read once per group).  The groups of a last,
//                 partial round are split along K into pieces whose partial
//                 sums the last piece adds in piece order.
//   down_rows_k : unit = (R rows of d, chunk of kPfChunk tokens); the chunk's
//                 y rows are summed in LDS over the experts in ascending
//                 order and written once -- no float atomics, deterministic.
// Units sharing weights (an expert's groups; a row block's token chunks) are
// placed on one XCD, where they meet in L2.
#include "pp_gateup.h"

namespace pp {
namespace {

struct DNParams {
    int T, d, E;
    const uint16_t *Wd;
    const uint16_t *h_hi;
    const uint16_t *h_lo;
    float *y;
    const float *bproj;    // [d] output bias, or NULL (0)
    const int32_t *cut;    // [E][ncut]: expert e's tokens below token c * kPfChunk
    int ncut;
    const int32_t *ebase;  // [E] first pair (h row) of each expert's bucket
    int tstride;           // toklist row stride per expert
    PlanView plan;
};

// Gate/up of one group (one expert, up to kPfGroupTokens of its tokens) in
// one workgroup, all 256 gate/up columns and all of K: wavefront w owns the
// expert's neuron tile w (16 neurons, gate and up) for every token tile of
// the group, so each weight fragment is read once per group, by one
// wavefront, straight from HBM into registers kPfPF K-steps ahead.  The
// group's token rows are staged in LDS in B-fragment order, kPfXC K-steps at
// a time: wavefront w copies token tile w's fragments of the next sub-chunk
// straight into LDS (buffer loads to LDS, no registers) while the current
// one is multiplied -- two LDS buffers, separate arrays so that the
// compiler's waits for the copies into one do not hold up reads of the
// other, and one barrier per sub-chunk.  Token tiles are multiplied in
// pairs, the pairs past the group skipped.  One workgroup per CU; the groups
// of one expert are neighbouring units on one XCD, where they share the
// expert's weights in L2.
constexpr int kPfXC = 8;                         // K-steps per staged token sub-chunk
constexpr int kPfPF = 4;                         // K-steps of weights in flight per wavefront
constexpr int kPfNT = kPfGroupTokens / 16;       // token tiles per group
static_assert(kPfXC % kPfPF == 0, "the weight ring restarts at every sub-chunk");
static_assert(kPfNT == kGuThreads / 64, "wavefront w stages token tile w");

// SiLU(a) * b with the hardware exp2 and reciprocal (about 1 ulp each):
// a / (1 + e^-a) = a * rcp(1 + 2^(-a log2 e)); a -> -inf gives 0, a -> +inf a.
__device__ __forceinline__ float silu_mul_fast(float a, float b) {
    const float t = __builtin_amdgcn_exp2f(-a * 1.44269504088896341f);
    return a * __builtin_amdgcn_rcpf(1.0f + t) * b;
}

// Copies 16 bytes per lane from the buffer into LDS: lane l's bytes land at
// dst + 16 l (dst wavefront-uniform).
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t r, uint4 *dst, unsigned off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        r, (__attribute__((address_space(3))) void *)dst, 16, off, 0, 0, 0);
}

template <bool GATED>
__device__ __forceinline__ float pf_act(const GUParams &P, int e, int r, float a, float b) {
    if (GATED) return silu_mul_fast(a, b);
    return act<false>(P, e, r, a, b);
}

// STREAM: a dense decode batch (every expert kept) streams the weights; a
// prefill group's weights are shared with the other groups of its expert in
// L2 and are read with plain loads.
template <bool GATED, bool STREAM>
__device__ __forceinline__ void pf_load_w(const uint16_t *wb, int s, uint4 &g, uint4 &u) {
    const uint16_t *p = wb + (size_t)s * kStepElems<GATED>;
    g = ldw16_if<STREAM>(p);
    if (GATED) u = ldw16_if<STREAM>(p + 512);
}

// Work list of gateup_pf_k with nG groups on nW workgroups: full rounds of
// whole groups (nW groups each), then the groups left over, each split into
// KS pieces along K (at most nW pieces in all, at most four per group), so
// that the last (or only) round uses more of the workgroups instead of
// leaving them idle.
struct PfSchedule {
    int full;    // groups run whole: [0, full)
    int KS;      // pieces per leftover group (1 when nothing is left over)
    int units;   // full + (nG - full) * KS
};

__device__ __forceinline__ PfSchedule pf_schedule(int nG, int nW, size_t part_rows) {
    PfSchedule S;
    S.full = nG - nG % nW;
    const int left = nG - S.full;
    S.KS = 1;
    if (left > 0) {
        S.KS = min(nW / left, 4);
        // each piece's partial rows (up to kPfGroupTokens per group) must fit
        while (S.KS > 1 && (size_t)left * S.KS * kPfGroupTokens > part_rows) --S.KS;
        if (S.KS < 1) S.KS = 1;
    }
    if (S.KS == 1) S.full = nG;
    S.units = S.full + (nG - S.full) * S.KS;
    return S;
}

// DEC: a decode batch whose groups come from the router's per-expert token
// masks (the decode plan, derived here in LDS as the decode gate/up kernel
// does; workgroup 0 stores it for the down projection).
template <bool GATED, bool DEC>
__global__ __launch_bounds__(kGuThreads, 1) void gateup_pf_k(GUParams P) {
    __shared__ uint4 xs0[kPfXC][kPfNT][64];
    __shared__ uint4 xs1[kPfXC][kPfNT][64];
    __shared__ int stok[kPfGroupTokens];
    __shared__ int s_flag;
    __shared__ DecodePlan D;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    if (DEC) decode_plan<true>(P, D, tid < P.E ? P.emask[tid] : 0ull);
    const int nG = DEC ? D.nG : P.plan.head[0];
    const int NS = P.NS, last = NS - 1;
    const int nsub = (NS + kPfXC - 1) / kPfXC;  // token sub-chunks over all of K
    const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
    const PfSchedule S = pf_schedule(nG, (int)gridDim.x, P.abpart_rows);
    const int slots_full = 8 * ((S.full + 7) / 8);
    for (int slot = blockIdx.x; slot < slots_full + (S.units - S.full); slot += gridDim.x) {
        // unit: a whole group (xcd-ordered, so an expert's groups share an
        // XCD), or piece `piece` of leftover group g (pieces of one group are
        // neighbouring slots)
        int g, piece = 0, KSg = 1;
        if (slot < slots_full) {
            g = xcd_order(slot, S.full);
            if (g >= S.full) continue;
        } else {
            const int v = slot - slots_full;
            g = S.full + v / S.KS;
            piece = v - (g - S.full) * S.KS;
            KSg = S.KS;
        }
        const int cA = piece * nsub / KSg, cB = (piece + 1) * nsub / KSg;
        const int sA = cA * kPfXC, sB = min(cB * kPfXC, NS);
        int e, n, p0;
        __syncthreads();  // the previous unit is done with stok and xs
        if (DEC) {
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
        const int nt = (n + 15) >> 4;
        const bool stager = wv < nt;
        // this lane's token row while staging tile wv (slots past the group
        // read its last token: they only feed output columns never stored)
        const unsigned xoff =
            ((unsigned)stok[min(16 * wv + (lane & 15), n - 1)] * (unsigned)P.d + 8u * (lane >> 4)) * 2u;
        const auto rx = buf_rsrc(P.x, stager ? (unsigned)((size_t)P.T * P.d * 2u) : 0u);
        const uint16_t *wb =
            P.Wgu + (size_t)(e * 8 + wv) * NS * kStepElems<GATED> + lane * 8;
        uint4 G[kPfPF], U[kPfPF];
#pragma unroll
        for (int i = 0; i < kPfPF; ++i) pf_load_w<GATED, DEC>(wb, min(sA + i, last), G[i], U[i]);
#pragma unroll
        for (int k = 0; k < kPfXC; ++k)
            lds_dma16(rx, &xs0[k][wv][0], xoff + (unsigned)min(sA + k, last) * kKStep * 2u);
        {
            const uint4 own = xs0[kPfXC - 1][wv][lane];  // waits for this wavefront's copies
            asm volatile("" ::"v"(own.x));
        }
        __syncthreads();
        f32x4 ag[kPfNT], au[kPfNT];
#pragma unroll
        for (int j = 0; j < kPfNT; ++j) {
            ag[j] = f32x4{0.f, 0.f, 0.f, 0.f};
            au[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        auto sub = [&](const uint4 (&cur)[kPfXC][kPfNT][64], uint4 (&nxt)[kPfXC][kPfNT][64], int s0) {
            const bool more = s0 + kPfXC < sB;
            if (more) {
#pragma unroll
                for (int k = 0; k < kPfXC; ++k)
                    lds_dma16(rx, &nxt[k][wv][0],
                              xoff + (unsigned)min(s0 + kPfXC + k, last) * kKStep * 2u);
            }
            // the token fragments of step k are read from LDS one step ahead
            uint4 b[kPfNT];
#pragma unroll
            for (int j = 0; j < kPfNT; ++j) b[j] = cur[0][j][lane];
#pragma unroll
            for (int k = 0; k < kPfXC; ++k) {
                uint4 bn[kPfNT];
                if (k + 1 < kPfXC) {
#pragma unroll
                    for (int j = 0; j < kPfNT; ++j) bn[j] = cur[k + 1][j][lane];
                }
                if (s0 + k < sB) {
                    // token tiles in pairs: the pairs past the group are skipped
#pragma unroll
                    for (int j = 0; j < kPfNT; ++j) {
                        if (j < 2 || nt > (j & ~1)) {
                            ag[j] = mfma16(G[k % kPfPF], b[j], ag[j]);
                            if (GATED) au[j] = mfma16(U[k % kPfPF], b[j], au[j]);
                        }
                    }
                }
                pf_load_w<GATED, DEC>(wb, min(s0 + k + kPfPF, last), G[k % kPfPF], U[k % kPfPF]);
                if (k + 1 < kPfXC) {
#pragma unroll
                    for (int j = 0; j < kPfNT; ++j) b[j] = bn[j];
                }
            }
            if (more) {
                // this wavefront's copies into nxt have landed before the barrier
                const uint4 own = nxt[kPfXC - 1][wv][lane];
                asm volatile("" ::"v"(own.x));
            }
            __syncthreads();
        };
        for (int s0 = sA; s0 < sB; s0 += 2 * kPfXC) {
            sub(xs0, xs1, s0);
            if (s0 + kPfXC < sB) sub(xs1, xs0, s0 + kPfXC);
        }
        // lane holds neurons r0 .. r0 + 3 of token slot 16 j + lane % 16
        const int r0 = wv * 16 + 4 * (lane >> 4);
        if (KSg > 1) {
            // a piece of a split group: its partial (a, b) in fragment order,
            // [piece][token tile][wavefront][a, b][lane] float4 (one KiB per
            // wavefront store); the last piece to arrive adds the pieces in
            // piece order at its own fragments and goes on to the epilogue
            constexpr unsigned kPieceBytes = kPfNT * 8 * 2 * 64 * 16;
            const auto pr = buf_rsrc(P.abpart + (size_t)(g - S.full) * KSg * (kPieceBytes / 4),
                                     (unsigned)KSg * kPieceBytes);
            const unsigned lo = ((unsigned)wv * 2 * 64 + lane) * 16;
#pragma unroll
            for (int j = 0; j < kPfNT; ++j) {
                if (j < nt) {
                    const unsigned o = (unsigned)piece * kPieceBytes + j * (8 * 2 * 64 * 16) + lo;
                    st_dev16(pr, o, ag[j]);
                    if (GATED) st_dev16(pr, o + 64 * 16, au[j]);
                }
            }
            if (!arrive_last(&P.cnt[g], (unsigned)KSg, &s_flag)) continue;
            f32x4 sa[kPfNT], su[kPfNT];
            for (int k = 0; k < KSg; ++k) {
#pragma unroll
                for (int j = 0; j < kPfNT; ++j) {
                    f32x4 va = ag[j], vu = au[j];
                    if (k != piece && j < nt) {
                        const unsigned o = (unsigned)k * kPieceBytes + j * (8 * 2 * 64 * 16) + lo;
                        va = ld_dev16(pr, o);
                        if (GATED) vu = ld_dev16(pr, o + 64 * 16);
                    }
                    sa[j] = k == 0 ? va : sa[j] + va;
                    su[j] = k == 0 ? vu : su[j] + vu;
                }
            }
#pragma unroll
            for (int j = 0; j < kPfNT; ++j) {
                ag[j] = sa[j];
                au[j] = su[j];
            }
        }
#pragma unroll
        for (int j = 0; j < kPfNT; ++j) {
            const int q = 16 * j + (lane & 15);
            if (j < nt && q < n) {
                const float scl = sig ? P.gsig[(size_t)stok[q] * P.E + e] : 1.0f;
                uint16_t hi[4], lo[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    split_bf16(pf_act<GATED>(P, e, r0 + i, ag[j][i], au[j][i]) * scl, hi[i],
                               lo[i]);
                const size_t row = (size_t)(p0 + q) * kExpertWidth + r0;
                *reinterpret_cast<uint2 *>(P.h_hi + row) = make_uint2(
                    hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16));
                *reinterpret_cast<uint2 *>(P.h_lo + row) = make_uint2(
                    lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16));
            }
        }
    }
}

// ------------------------------------------------------------------ prefill

__global__ __launch_bounds__(256) void dispatch_k(const uint32_t *__restrict__ selmask, int T,
                                                  int E, int32_t *__restrict__ ecount,
                                                  int32_t *__restrict__ tokl, int stride,
                                                  int32_t *__restrict__ cut, int ncut,
                                                  int32_t *__restrict__ ebase, uint32_t *cnt,
                                                  PlanView plan, int num_cu) {
    static_assert(kPfChunk % 256 == 0, "chunk starts fall on blocks of 256 tokens");
    constexpr int kBlocks = 8;  // blocks of 256 tokens whose flags are loaded at once
    __shared__ int scan[8];
    __shared__ __align__(16) int wc[2][kBlocks][4];  // per block and wavefront: tokens that kept e
    __shared__ int s_flag;
    const int e = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int w = e >> 5, b = e & 31;
    const unsigned long long below = (1ull << lane) - 1ull;
    int base = 0, par = 0;
    for (int T0 = 0; T0 < T; T0 += kBlocks * 256, par ^= 1) {
        uint32_t word[kBlocks];
#pragma unroll
        for (int j = 0; j < kBlocks; ++j) {
            const int t = T0 + 256 * j + tid;
            word[j] = t < T ? selmask[(size_t)t * 8 + w] : 0u;
        }
        unsigned long long bal[kBlocks];
#pragma unroll
        for (int j = 0; j < kBlocks; ++j) {
            bal[j] = __ballot((word[j] >> b) & 1u);
            if (lane == 0) wc[par][j][wv] = __popcll(bal[j]);
        }
        __syncthreads();
        // block j's tokens follow those of blocks 0 .. j - 1, in token order
#pragma unroll
        for (int j = 0; j < kBlocks; ++j) {
            const int t = T0 + 256 * j + tid;
            const int4 c = *reinterpret_cast<const int4 *>(wc[par][j]);
            const int before = (wv > 0 ? c.x : 0) + (wv > 1 ? c.y : 0) + (wv > 2 ? c.z : 0);
            if (tid == 0 && T0 + 256 * j < T && (T0 + 256 * j) % kPfChunk == 0)
                cut[(size_t)e * ncut + (T0 + 256 * j) / kPfChunk] = base;
            if ((bal[j] >> lane) & 1ull)
                tokl[(size_t)e * stride + base + before + __popcll(bal[j] & below)] = t;
            base += (c.x + c.y) + (c.z + c.w);
        }
    }
    if (tid == 0) {
        cut[(size_t)e * ncut + (T + kPfChunk - 1) / kPfChunk] = base;
        st_dev_u32(reinterpret_cast<uint32_t *>(ecount + e), (uint32_t)base);
    }
    if (!arrive_last(cnt, (unsigned)E, &s_flag)) return;
    // prefill plan: expert e's bucket becomes ceil(c_e / gs) groups of nearly
    // equal size (the first c_e % groups one token larger), so that the groups
    // of one expert stream its weights at the same pace and meet in L2.  The
    // group size gs is the smallest of 64, 80, 96, 112 whose groups all fit in
    // one round on the CUs (smaller groups stage fewer token rows and spread
    // over more CUs), else kPfGroupTokens.
    const int c = (tid < E) ? (int)ld_dev_u32(reinterpret_cast<uint32_t *>(ecount + tid)) : 0;
    int gs = kPfGroupTokens;
    if ((long)T * E / 64 + E < 65535) {
        // the four sizes' group counts, two to an int (each sum below 2^16): one scan
        int x0, x1, p0, p1;
        block_excl_scan2(((c + 63) / 64) | (((c + 79) / 80) << 16),
                         ((c + 95) / 96) | (((c + 111) / 112) << 16), &x0, &x1, &p0, &p1, scan);
        const int n64 = p0 & 0xFFFF, n80 = p0 >> 16, n96 = p1 & 0xFFFF, n112 = p1 >> 16;
        gs = n64 <= num_cu ? 64 : n80 <= num_cu ? 80 : n96 <= num_cu ? 96 : n112 <= num_cu ? 112 : gs;
    }
    const int nch = (c + gs - 1) / gs;
    int cb, off, nG, npairs;
    block_excl_scan2(nch, c, &cb, &off, &nG, &npairs, scan);
    if (tid < E) {
        plan.egrp[tid] = cb;
        ebase[tid] = off;
    }
    if (tid == 0) plan.egrp[E] = nG;
    const int gbase = nch > 0 ? c / nch : 0, grem = nch > 0 ? c - gbase * nch : 0;
    for (int ch = 0, first = 0; ch < nch; ++ch) {
        const int g = cb + ch, n = gbase + (ch < grem ? 1 : 0);
        plan.grp_e[g] = tid;
        plan.grp_pair[g] = off + first;
        plan.grp_n[g] = n;
        plan.grp_tok[g] = tid * stride + first;
        first += n;
    }
    if (tid == 0) {
        plan.head[0] = nG;
        plan.head[1] = npairs;
    }
}

// Unit = (R rows of d, a chunk of kPfChunk consecutive tokens).  The chunk's
// outputs in those rows stay in LDS for the whole unit, starting from the
// output bias (or 0).  The experts are taken in ascending order; the tokens
// of the chunk that kept expert e are a contiguous run of its ascending
// bucket (positions cut[e][c] .. cut[e][c + 1]), so their h rows are
// consecutive.  A step is one expert's R x 128 down block, staged in LDS, and
// up to eight 16-token tiles of its run, one per wavefront (bf16 MFMA
// 16x16x32: A = the down block, B = the tokens' h, hi then lo per K-step);
// each tile is added to its tokens' LDS rows, and barriers separate the
// steps.  Every output is thus the bias plus its token's pair contributions
// in ascending expert order -- deterministic, with no atomics and no per-pair
// rows in memory.  Every step issues the same loads (bounds-checked buffer
// loads: lanes past the run read zeros without touching memory), kRowAhead
// steps ahead, so each wait is for one step's data only.  The token chunks of
// one row block are neighbouring units, placed on one XCD, so they share the
// down blocks in L2.
constexpr int kRowAhead = 3;  // steps whose loads are in flight


template <int R>
struct DownRowsLds {
    float y[kPfChunk * (R + 4)];  // [token][row], rows padded by 4 floats
    u32x4_t w[R / 16 * 4 * 64];   // [row tile][K-step][lane]: A fragments
    int4 ent[kMaxExperts];        // experts with tokens in the chunk, ascending:
                                  // (expert, tokens in the run, first pair (h row)
                                  // of the run, its first bucket position)
    int m, steps;
};

// One step's loads as held by a thread, with the step's (wavefront-uniform)
// description: list entry k (m past the list), tokens n of its run and the
// first place t16 of the wavefront's tile in the run.
struct RowStep {
    u32x4_t w0, w1;         // its share of the down block (R = 64: both)
    u32x4_t bh[4], bl[4];   // the wavefront's tile: h hi / lo B fragments
    unsigned tok;           // token of the lane's slot (0 past the run)
    int k, n, t16;
};

// Steps in order: list entry k, round r (tiles 8 r .. 8 r + 7 of its run).
// The cursor carries its entry and the next one (read one step ahead), so
// moving on needs no LDS round trip.
struct RowCursor {
    int k, r;
    int4 cur, next;
};

template <int R>
__device__ __forceinline__ void rows_next(RowCursor &c, const DownRowsLds<R> &S, int m) {
    if (c.k < m && 8 * 16 * (c.r + 1) < c.cur.y) {
        ++c.r;
    } else {
        ++c.k;
        c.r = 0;
        c.cur = c.next;
        c.next = S.ent[min(c.k + 1, m - 1)];
    }
}

// Issues step c's loads (past the list: all out of range, zeros).
template <int R>
__device__ __forceinline__ void rows_issue(RowStep &st, const DNParams &P, const RowCursor &c,
                                           int m, int rb, int tid) {
    constexpr int MT = R / 16, WN = MT * 4 * 64;
    static_assert(WN <= 2 * 512, "at most two uint4 of a down block per thread");
    // every descriptor operand is wavefront-uniform, so it lives in SGPRs
    const int lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ck = __builtin_amdgcn_readfirstlane(c.k), cr = __builtin_amdgcn_readfirstlane(c.r);
    const bool live = ck < m;
    const int e = __builtin_amdgcn_readfirstlane(c.cur.x);
    const int n = live ? __builtin_amdgcn_readfirstlane(c.cur.y) : 0;
    const int p0 = __builtin_amdgcn_readfirstlane(c.cur.z);
    const int a0 = __builtin_amdgcn_readfirstlane(c.cur.w);
    const int t16 = 16 * (wv + 8 * cr);       // the tile's first place in the run
    const int nt = max(0, min(16, n - t16));  // tokens in the tile
    st.k = live ? ck : m;
    st.n = n;
    st.t16 = t16;
    // down block: contiguous WN uint4
    const auto rw = buf_rsrc(P.Wd + ((size_t)e * (P.d / 16) + (size_t)rb * MT) * 256 * 8,
                              live ? WN * 16u : 0u);
    st.w0 = __builtin_amdgcn_raw_buffer_load_b128(rw, (unsigned)tid * 16u, 0, 0);
    if (WN > 512) st.w1 = __builtin_amdgcn_raw_buffer_load_b128(rw, (unsigned)(512 + tid) * 16u, 0, 0);
    // the tile's h rows and tokens
    const size_t q0 = (size_t)p0 + t16;
    const auto rh = buf_rsrc(P.h_hi + q0 * kExpertWidth, (unsigned)nt * kExpertWidth * 2u);
    const auto rl = buf_rsrc(P.h_lo + q0 * kExpertWidth, (unsigned)nt * kExpertWidth * 2u);
    const unsigned o = ((unsigned)(lane & 15) * kExpertWidth + 8u * (lane >> 4)) * 2u;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        st.bh[s] = __builtin_amdgcn_raw_buffer_load_b128(rh, o + s * kKStep * 2u, 0, 0);
        st.bl[s] = __builtin_amdgcn_raw_buffer_load_b128(rl, o + s * kKStep * 2u, 0, 0);
    }
    const auto rt = buf_rsrc(P.plan.toklist + (size_t)e * P.tstride + a0 + t16, (unsigned)nt * 4u);
    st.tok = __builtin_amdgcn_raw_buffer_load_b32(rt, (unsigned)(lane & 15) * 4u, 0, 0);
}

// Runs step st: its down block to LDS, then the wavefront's tile.
template <int R>
__device__ __forceinline__ void rows_run(DownRowsLds<R> &S, const RowStep &st, int m, int t0,
                                         int tid) {
    constexpr int MT = R / 16, YS = R + 4, WN = MT * 4 * 64;
    const int lane = tid & 63;
    __syncthreads();  // the previous step's block and rows are done with
    if (WN >= 512 || tid < WN) S.w[tid] = st.w0;
    if (WN > 512) S.w[512 + tid] = st.w1;
    __syncthreads();
    const int k = __builtin_amdgcn_readfirstlane(st.k), n = __builtin_amdgcn_readfirstlane(st.n);
    const int t16 = __builtin_amdgcn_readfirstlane(st.t16);
    if (k >= m || t16 >= n) return;
    // lane: rows 4 (lane / 16) + i of each row tile, its slot's token.  The
    // rows and all of the down block's fragments are read from LDS first (the
    // barrier ordered the reads after the previous step's adds), then the
    // products run back to back.
    const bool own = t16 + (lane & 15) < n;
    float *yr = &S.y[(own ? (int)st.tok - t0 : 0) * YS + 4 * (lane >> 4)];
    float4 yv[MT];
    uint4 a[MT][4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            a[mt][s] = *reinterpret_cast<const uint4 *>(&S.w[(mt * 4 + s) * 64 + lane]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) yv[mt] = *reinterpret_cast<const float4 *>(yr + 16 * mt);
    __builtin_amdgcn_sched_barrier(0);
    f32x4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const uint4 bh = *reinterpret_cast<const uint4 *>(&st.bh[s]);
        const uint4 bl = *reinterpret_cast<const uint4 *>(&st.bl[s]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            acc[mt] = mfma16(a[mt][s], bh, acc[mt]);
            acc[mt] = mfma16(a[mt][s], bl, acc[mt]);
        }
    }
    if (own) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            float4 v = yv[mt];
            v.x += acc[mt][0];
            v.y += acc[mt][1];
            v.z += acc[mt][2];
            v.w += acc[mt][3];
            *reinterpret_cast<float4 *>(yr + 16 * mt) = v;
        }
    }
}

template <int R>
__global__ __launch_bounds__(512, 1) void down_rows_k(DNParams P) {
    constexpr int YS = R + 4;  // LDS row stride of y in floats
    __shared__ DownRowsLds<R> S;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int nC = (P.T + kPfChunk - 1) / kPfChunk;
    const int units = (P.d / R) * nC;
    const int slots = 8 * ((units + 7) / 8);
    for (int slot = blockIdx.x; slot < slots; slot += gridDim.x) {
        const int unit = xcd_order(slot, units);
        if (unit >= units) continue;
        const int rb = unit / nC, c = unit - rb * nC;
        const int t0 = c * kPfChunk, nt = min(kPfChunk, P.T - t0);
        if (wv == 0) {
            int m = 0, steps = 0;
            for (int e0 = 0; e0 < P.E; e0 += 64) {
                const int e = e0 + lane;
                int a = 0, b = 0;
                if (e < P.E) {
                    a = P.cut[(size_t)e * P.ncut + c];
                    b = P.cut[(size_t)e * P.ncut + c + 1];
                }
                const unsigned long long bal = __ballot(b > a);
                if (b > a)
                    S.ent[m + __popcll(bal & ((1ull << lane) - 1ull))] =
                        make_int4(e, b - a, P.ebase[e] + a, a);
                m += __popcll(bal);
                const int rounds = b > a ? (b - a + 127) / 128 : 0;
                steps += __builtin_amdgcn_readlane(wave_scan_i32(rounds), 63);
            }
            if (lane == 0) {
                S.m = m;
                S.steps = steps;
            }
        }
        for (int i = tid; i < nt * (R / 4); i += 512) {
            const int t = i / (R / 4), q = i - t * (R / 4);
            *reinterpret_cast<float4 *>(&S.y[t * YS + 4 * q]) =
                P.bproj ? *reinterpret_cast<const float4 *>(P.bproj + rb * R + 4 * q)
                        : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        __syncthreads();
        const int m = S.m, steps = S.steps;
        if (m > 0) {
            RowStep st[kRowAhead];
            RowCursor ci = {0, 0, S.ent[0], S.ent[min(1, m - 1)]};  // next step to issue
#pragma unroll
            for (int i = 0; i < kRowAhead; ++i) {
                rows_issue<R>(st[i], P, ci, m, rb, tid);
                rows_next<R>(ci, S, m);
            }
            for (int s0 = 0; s0 < steps; s0 += kRowAhead) {
#pragma unroll
                for (int i = 0; i < kRowAhead; ++i) {
                    rows_run<R>(S, st[i], m, t0, tid);
                    rows_issue<R>(st[i], P, ci, m, rb, tid);
                    rows_next<R>(ci, S, m);
                }
            }
        }
        __syncthreads();
        for (int i = tid; i < nt * (R / 4); i += 512) {
            const int t = i / (R / 4), q = i - t * (R / 4);
            *reinterpret_cast<float4 *>(P.y + (size_t)(t0 + t) * P.d + rb * R + 4 * q) =
                *reinterpret_cast<const float4 *>(&S.y[t * YS + 4 * q]);
        }
        __syncthreads();
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
    P.bproj = L->bproj;
    P.cut = L->pf_cut;
    P.ncut = L->pf_ncut;
    P.ebase = L->pf_ebase;
    P.tstride = L->max_tokens;
    P.plan = plan_view(L, true);
    return P;
}

}  // namespace

// Gate/up of a decode batch in which every token keeps every expert (dense):
// the grouped kernel above, its groups from the decode plan.
void launch_gateup_dense_dec(pp_layer *L, const uint16_t *x, int T, hipStream_t s) {
    const GUParams gp = gu_params(L, x, T, false);
    if (L->gated)
        hipLaunchKernelGGL((gateup_pf_k<true, true>), dim3(L->num_cu), dim3(kGuThreads), 0, s, gp);
    else
        hipLaunchKernelGGL((gateup_pf_k<false, true>), dim3(L->num_cu), dim3(kGuThreads), 0, s, gp);
}

counter_layout counters_for(const pp_dims &dm, int max_tokens) {
    counter_layout c;
    c.route = 0;
    c.gateup = (size_t)plan_max_groups(dm, max_tokens);
    c.down = (size_t)((dm.d + 127) / 128);
    c.dispatch = 1;
    c.total = c.route + c.gateup + c.down + c.dispatch;
    return c;
}

hipError_t launch_prefill_ffn(pp_layer *L, const uint16_t *x, int T, float *y, hipStream_t s) {
    const pp_dims &dm = L->dm;
    const counter_layout cl = counters_for(dm, L->max_tokens);
    prof_mark(L, PP_KERNEL_DISPATCH, s, true);
    hipLaunchKernelGGL(dispatch_k, dim3(dm.E), dim3(256), 0, s, L->selmask, T, dm.E, L->ecount,
                       L->tokl, L->max_tokens, L->pf_cut, L->pf_ncut, L->pf_ebase,
                       L->counters + cl.dispatch_base(), plan_view(L, true), L->num_cu);
    prof_mark(L, PP_KERNEL_DISPATCH, s, false);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const GUParams gp = gu_params(L, x, T, true);
    prof_mark(L, PP_KERNEL_GATEUP, s, true);
    // one workgroup per CU (the kernel's registers and LDS allow no more)
    if (L->gated)
        hipLaunchKernelGGL((gateup_pf_k<true, false>), dim3(L->num_cu), dim3(kGuThreads), 0, s, gp);
    else
        hipLaunchKernelGGL((gateup_pf_k<false, false>), dim3(L->num_cu), dim3(kGuThreads), 0, s, gp);
    prof_mark(L, PP_KERNEL_GATEUP, s, false);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    const DNParams dp = dn_params(L, T, y);
    // the widest row block (64, 32 or 16 rows) that still gives every CU a unit
    const int nC = (T + kPfChunk - 1) / kPfChunk;
    const int R = (dm.d / 64) * nC >= L->num_cu ? 64 : ((dm.d / 32) * nC >= L->num_cu ? 32 : 16);
    static const int occ64 = resident(down_rows_k<64>, 512);
    static const int occ32 = resident(down_rows_k<32>, 512);
    static const int occ16 = resident(down_rows_k<16>, 512);
    prof_mark(L, PP_KERNEL_DOWN, s, true);
    if (R == 64)
        hipLaunchKernelGGL(down_rows_k<64>, dim3(occ64 * L->num_cu), dim3(512), 0, s, dp);
    else if (R == 32)
        hipLaunchKernelGGL(down_rows_k<32>, dim3(occ32 * L->num_cu), dim3(512), 0, s, dp);
    else
        hipLaunchKernelGGL(down_rows_k<16>, dim3(occ16 * L->num_cu), dim3(512), 0, s, dp);
    prof_mark(L, PP_KERNEL_DOWN, s, false);
    return hipGetLastError();
}

}  // namespace pp
