// Decode expert evaluation (T <= 64): Eq. (ffn) restricted to the batch's
// kept experts and summed per token, Eqs. (moefication_decomp), (moe_output).
//
// The plan has one group per expert kept by at least one token of the batch:
// every gate/up workgroup derives it from the router's per-expert token masks
// and workgroup 0 stores it for the down projection.
//
//   gateup_dec_k: the gate/up projections and the SiLU product of every
//                 group (or the non-gated layer's input projection, bias and
//                 GELU).  Neuron-tile units: unit = one 16-neuron tile of one
//                 kept expert over all of K (at most 32 of its tokens), its K
//                 in 2, 4 or 8 parts on as many wavefronts (more parts the
//                 fewer tiles the call has), the parts summed in LDS, so no
//                 partial sums pass between workgroups.  Small unions with
//                 many tokens per group: unit = (group, K-slice) with the
//                 tokens staged in LDS (code shared with prefill); the K-split
//                 (one slice more for some groups) makes the units fill the
//                 resident workgroups exactly, one round.
//   down_dec_k  : sparse groups (<= 16 tokens per group on average): unit = one
//                 16-row tile of d over all groups; each of the 8 wavefronts
//                 takes every eighth group, tile by tile of 16 tokens (three
//                 in flight), multiplies the 16x128 down block with the tokens'
//                 h (two MFMAs per fragment: hi and lo) and adds into its own
//                 LDS accumulator [tokens][16 rows]; the accumulators are
//                 summed in wavefront order and y written once.
//                 Dense groups: unit = (128 rows, chunk of groups), h staged
//                 once in LDS for all 8 wavefronts, chunk partials summed in
//                 chunk order by the last chunk to arrive.
//   down_dense_k: every token keeps every expert (16-64 tokens): outputs
//                 accumulate in registers across a unit's experts, h copied
//                 into LDS two experts ahead; dense_sum_k (its own launch)
//                 sums the expert chunks' partials in chunk order.
//                 No float atomics: decode is deterministic.
#include "pp_gateup.h"

namespace pp {
namespace {

constexpr int kDnThreads = 512;    // down projection: 8 wavefronts per workgroup
constexpr int kDnR = 1;            // 16-row tiles per down item (sparse groups)
constexpr int kDnRing = 4;         // sparse groups: items per wavefront ring (three in flight)
constexpr int kShRows = 128;       // dense groups: rows per unit (8 wavefronts x 16)
constexpr int kShYS = kShRows + 4;
constexpr int kShTiles = kDecodeTile / 16;

struct DNParams {
    int T, d, E;
    const uint16_t *Wd;
    const uint16_t *h_hi;
    const uint16_t *h_lo;
    float *y;
    const float *bproj;  // [d] output bias added once per token, or NULL
    float *ypart;      // [kDecodeChunks][T][d] chunk partials (dense groups)
    uint32_t *dn_cnt;  // [ceil(d / 128)] chunk arrivals per row block
    PlanView plan;
};

// ------------------------------------------------------------------ gate/up

// Neuron-tile units (sparse groups): unit = one 16-neuron tile of one group's
// expert over all of K, taken by PARTS wavefronts of the workgroup -- two
// when the union fills the chip (each wavefront then streams half of the
// tile's K: long streams keep more of HBM busy than more, shorter ones), all
// eight for a small union (a latency-bound unit is done sooner in eight
// parts); wavefront q of the unit takes K part q, its token B fragments
// straight from x (a few tokens, cache resident), the weights PF steps ahead
// in two register buffers.  The parts' (a, b) are added in LDS in part order
// and the unit writes h for its 16 neurons: no partial sums leave the
// workgroup, so no hand-off between workgroups.
constexpr int kTileSlots = 4;       // units per workgroup at a time (two-part units)
constexpr int kTileParts = 2;       // wavefronts per unit (K parts) when the union fills the chip
constexpr int kTilePF = 2;          // K-steps per register buffer (two buffers)
constexpr int kTileMaxNT = 2;       // token tiles per unit (batches of up to 32 tokens)
static_assert(kTileSlots * kTileParts * 64 == kGuThreads, "four slots of two wavefronts");
static_assert(kTileSlots * kTileMaxNT * 2 * kTileParts * 64 * 16 <= kXBufBytes,
              "the parts' (a, b) of all slots fit in the token staging buffer");

template <int NT, bool GATED, int PF, bool STREAM>
__device__ __forceinline__ void tile_load(const uint16_t *wb, const uint16_t *const (&xr)[NT],
                                          int step, int last, uint4 (&G)[PF], uint4 (&U)[PF],
                                          uint4 (&B)[PF][NT]) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
        const int s = min(step + i, last);
        const uint16_t *p = wb + (size_t)s * kStepElems<GATED>;
        G[i] = ldw16_if<STREAM>(p);
        if (GATED) U[i] = ldw16_if<STREAM>(p + 512);
#pragma unroll
        for (int j = 0; j < NT; ++j) B[i][j] = ldg16(xr[j] + s * kKStep);
    }
}

template <int NT, bool GATED, int PF>
__device__ __forceinline__ void tile_mfma(int nvalid, const uint4 (&G)[PF], const uint4 (&U)[PF],
                                          const uint4 (&B)[PF][NT], f32x4 (&ag)[NT],
                                          f32x4 (&au)[NT]) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
        if (i < nvalid) {
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                ag[j] = mfma16(G[i], B[i][j], ag[j]);
                if (GATED) au[j] = mfma16(U[i], B[i][j], au[j]);
            }
        }
    }
}

// One wavefront's K part q (of PARTS) of a tile unit; leaves its (a, b) in red.
template <int NT, bool GATED, int PF, int PARTS, bool STREAM>
__device__ __forceinline__ void tile_part(const GUParams &P, int e, int nt, int n,
                                          const int *tok, int q, int lane, float4 *red) {
    const int sA = q * P.NS / PARTS, sB = (q + 1) * P.NS / PARTS;
    const uint16_t *wb = P.Wgu + (size_t)(e * 8 + nt) * P.NS * kStepElems<GATED> + lane * 8;
    const uint16_t *xr[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int slot = 16 * j + (lane & 15);
        // an empty slot reads the group's first token: it only feeds that
        // slot's output column, which is never stored
        xr[j] = P.x + (size_t)tok[slot < n ? slot : 0] * P.d + 8 * (lane >> 4);
    }
    f32x4 ag[NT], au[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        ag[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        au[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int last = sB - 1;
    uint4 G0[PF], U0[PF], G1[PF], U1[PF], B0[PF][NT], B1[PF][NT];
    if (sA < sB) tile_load<NT, GATED, PF, STREAM>(wb, xr, sA, last, G0, U0, B0);  // small d: a part may be empty
    for (int s = sA; s < sB; s += 2 * PF) {
        if (s + PF < sB) tile_load<NT, GATED, PF, STREAM>(wb, xr, s + PF, last, G1, U1, B1);
        tile_mfma<NT, GATED, PF>(min(PF, sB - s), G0, U0, B0, ag, au);
        if (s + 2 * PF < sB) tile_load<NT, GATED, PF, STREAM>(wb, xr, s + 2 * PF, last, G0, U0, B0);
        if (s + PF < sB) tile_mfma<NT, GATED, PF>(min(PF, sB - s - PF), G1, U1, B1, ag, au);
    }
    // red[(j * 2 + {a, b}) * PARTS + q][lane]
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        red[((j * 2 + 0) * PARTS + q) * 64 + lane] = make_float4(ag[j][0], ag[j][1], ag[j][2], ag[j][3]);
        red[((j * 2 + 1) * PARTS + q) * 64 + lane] = make_float4(au[j][0], au[j][1], au[j][2], au[j][3]);
    }
}

// h of a tile unit from its PARTS K parts, summed in part order; wavefront j
// of the unit takes token tile j.
template <int NT, bool GATED, int PARTS>
__device__ __forceinline__ void tile_epilogue(const GUParams &P, int e, int nt, int n, int p0,
                                              const int *tok, int j, int lane, const float4 *red) {
    const int qs = 16 * j + (lane & 15);
    if (j >= NT || qs >= n) return;
    float4 a = red[((j * 2 + 0) * PARTS + 0) * 64 + lane];
    float4 b = red[((j * 2 + 1) * PARTS + 0) * 64 + lane];
#pragma unroll
    for (int q = 1; q < PARTS; ++q) {
        const float4 pa = red[((j * 2 + 0) * PARTS + q) * 64 + lane];
        const float4 pb = red[((j * 2 + 1) * PARTS + q) * 64 + lane];
        a.x += pa.x; a.y += pa.y; a.z += pa.z; a.w += pa.w;
        b.x += pb.x; b.y += pb.y; b.z += pb.z; b.w += pb.w;
    }
    const bool sig = (P.flags & PP_AGG_SIGMOID) != 0;
    const float scl = sig ? P.gsig[(size_t)tok[qs] * P.E + e] : 1.0f;
    const int r0 = nt * 16 + 4 * (lane >> 4);
    const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
    uint16_t hi[4], lo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) split_bf16(act<GATED>(P, e, r0 + i, av[i], bv[i]) * scl, hi[i], lo[i]);
    const size_t row = (size_t)(p0 + qs) * kExpertWidth + r0;
    *reinterpret_cast<uint2 *>(P.h_hi + row) =
        make_uint2(hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16));
    *reinterpret_cast<uint2 *>(P.h_lo + row) =
        make_uint2(lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16));
}

// Sum of one int per thread over the kGuThreads threads, returned to every
// thread; `sm` (16-byte aligned) holds one int per wavefront and is free
// again after the caller's next barrier.
__device__ __forceinline__ int block_sum(int v, int *sm) {
    static_assert(kGuThreads == 512, "eight wavefront sums, read as two int4");
    const int wv = threadIdx.x >> 6;
    const int w = __builtin_amdgcn_readlane(wave_scan_i32(v), 63);
    if ((threadIdx.x & 63) == 0) sm[wv] = w;
    __syncthreads();
    const int4 a = reinterpret_cast<const int4 *>(sm)[0], b = reinterpret_cast<const int4 *>(sm)[1];
    return ((a.x + a.y) + (a.z + a.w)) + ((b.x + b.y) + (b.z + b.w));
}

// Position of the n-th (from 0) set bit of w, which has more than n set bits.
__device__ __forceinline__ int nth_set_bit(unsigned long long w, int n) {
    int pos = 0;
#pragma unroll
    for (int sh = 32; sh >= 1; sh >>= 1) {
        const int c = __popcll(w & ((1ull << sh) - 1ull));
        if (n >= c) {
            n -= c;
            w >>= sh;
            pos += sh;
        }
    }
    return pos;
}

// Tile units without the batch plan: the kept experts come as bitmask words
// (word i: experts 64 i .. 64 i + 63), unit u is tile u % 8 of the
// (u / 8)-th kept expert, found by popcounts, so a workgroup's weights
// stream once it has the words; the unit's first pair row (tokens of the
// kept experts before it) is a wavefront sum of mask popcounts at the end,
// and workgroup 0 stores the batch plan for the down projection after its
// units.  A unit takes PARTS wavefronts (K parts), so a workgroup holds
// 8 / PARTS units at a time: slot h of workgroup b takes units b + h * grid,
// then the next (8 / PARTS) * grid, ... (every workgroup one unit before any
// takes two); barriers stay outside the per-unit work, so every wavefront
// meets them whether or not it holds a unit.  A unit of a group with more than 16
// tokens takes two token tiles (and one K-step per register buffer, which
// keeps the kernel within its registers).  Units 8 nG .. 8 (nG + nBig) - 1
// take the tokens past the first 32 of the nBig experts kept by more than 32
// tokens (bitmask words `big`): u - 8 nG is tile (u - 8 nG) % 8 of the
// ((u - 8 nG) / 8)-th of them, so no unit holds more than 32 tokens.
template <bool GATED, int PARTS, bool STREAM>
__device__ void tile_units_bits(const GUParams &P, DecodePlan &D, unsigned long long m_own,
                                const unsigned long long *s_mask,
                                const unsigned long long *kept, int nG, int *tokh, float4 *red,
                                const unsigned long long *big, int nBig) {
    constexpr int SLOTS = (kGuThreads / 64) / PARTS;  // units per workgroup at a time
    static_assert(SLOTS * PARTS == kGuThreads / 64 && SLOTS <= kTileSlots, "whole wavefronts");
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int slot = wv / PARTS, q = wv % PARTS;
    const int units = (nG + nBig) * 8, grid = (int)gridDim.x;
    int *tok = tokh + slot * kGroupTokens;
    float4 *rh = red + slot * (kTileMaxNT * 2 * PARTS * 64);
    for (int base = 0; base < units; base += SLOTS * grid) {
        const int u = base + slot * grid + (int)blockIdx.x;
        const bool act = u < units;
        // units past 8 nG: the tokens past the first 32 of the experts kept by
        // more than 32 tokens (words `big`), in expert order
        const bool second = u >= nG * 8;
        const unsigned long long *words = second ? big : kept;
        int g = act ? (second ? u - nG * 8 : u) >> 3 : 0, wi = 0;
        while (wi < kMaxExperts / 64 - 1 && g >= __popcll(words[wi])) g -= __popcll(words[wi++]);
        const int e = act ? 64 * wi + nth_set_bit(words[wi], g) : 0, nt = u & 7;
        const unsigned long long mall = s_mask[e];
        // the unit's tokens: the first 32 of the expert's (all, for 32 or
        // fewer), or those past them
        const int nall = __popcll(mall), t0 = second ? 32 : 0;
        const int n = second ? nall - 32 : min(nall, 32);
        if (act && q == 0 && ((mall >> lane) & 1ull)) {
            const int r = __popcll(mall & ((1ull << lane) - 1ull)) - t0;
            if (r >= 0 && r < 32) tok[r] = lane;
        }
        __syncthreads();
        if (act) {
            if (n <= 16)
                tile_part<1, GATED, kTilePF, PARTS, STREAM>(P, e, nt, n, tok, q, lane, rh);
            else
                tile_part<2, GATED, 1, PARTS, STREAM>(P, e, nt, n, tok, q, lane, rh);
        }
        __syncthreads();
        if (act && q < ((n + 15) >> 4)) {
            int c = 0;
            for (int e2 = lane; e2 < e; e2 += 64) c += __popcll(s_mask[e2]);
            const int p0 = __builtin_amdgcn_readlane(wave_scan_i32(c), 63) + t0;
            if (n <= 16)
                tile_epilogue<1, GATED, PARTS>(P, e, nt, n, p0, tok, q, lane, rh);
            else
                tile_epilogue<2, GATED, PARTS>(P, e, nt, n, p0, tok, q, lane, rh);
        }
        __syncthreads();
    }
    if (blockIdx.x == 0) decode_plan<true>(P, D, m_own);
}

template <bool GATED, int NTMAX, int PF>
__global__ __launch_bounds__(kGuThreads, 4) void gateup_dec_k(GUParams P) {
    static_assert(kGuThreads == kSelThreads, "the selection runs on the whole workgroup");
    __shared__ union {
        uint4 xf[kXBufBytes / 16];
        SelLds<1> sel;  // the single-token selection, before any token is staged
    } U;
    uint4 *const xf = U.xf;
    __shared__ int stok[kTileSlots * kGroupTokens];
    __shared__ int s_flag;
    __shared__ DecodePlan D;
    __shared__ unsigned long long s_mask[kMaxExperts];
    __shared__ unsigned long long s_kept[kMaxExperts / 64];
    __shared__ unsigned long long s_big[kMaxExperts / 64];
    __shared__ __align__(16) int s_sum[kGuThreads / 64];
    __shared__ float s_gsig[kMaxExperts];
    const int tid = threadIdx.x;
    unsigned long long m_own;
    if (P.select_here) {
        // single-token decode: every workgroup selects the token's experts
        // from the partial logits (the same arithmetic as the router's
        // selection kernel, so the same bits); workgroup 0 stores the
        // selection outputs, and the gate weights the epilogues scale by
        // come from LDS
        const SelOut r = select_tokens<1>(P.rp, 0, U.sel);
        if (blockIdx.x == 0) select_store<1>(P.rp, U.sel, r);
        const bool kept = tid < P.E && r.rank < r.k;
        m_own = kept ? 1ull : 0ull;
        if (tid < P.E)
            s_gsig[tid] = (P.flags & PP_AGG_SIGMOID) ? r.sg : 1.0f;
        P.gsig = s_gsig;
        __syncthreads();  // the selection's scratch is done with
    } else {
        m_own = tid < P.E ? P.emask[tid] : 0ull;
    }
    if (tid < kMaxExperts) s_mask[tid] = m_own;
    {
        const unsigned long long kb = __ballot(m_own != 0ull);
        const unsigned long long bb = __ballot(__popcll(m_own) > 32);
        if (tid < kMaxExperts && (tid & 63) == 0) {
            s_kept[tid >> 6] = kb;
            s_big[tid >> 6] = bb;
        }
    }
    const int grid = (int)gridDim.x;
    // At least one neuron tile per workgroup: neuron-tile units, no K split,
    // every unit of the call in flight at once (up to kTileSlots per
    // workgroup).  A unit takes at most 32 tokens (two token tiles, read from
    // x directly): an expert kept by more has a second set of tile units for
    // its tokens past the first 32.  (With fewer tiles than workgroups, the
    // units' long streams would leave most of the chip idle: such calls take
    // four-part units, and small unions eight-part units, below.)
    {
        // kept experts and pairs in one block sum: (pairs << 10) + experts,
        // whether a group spans more than two token tiles, and how many do
        const int over32 = NTMAX > 2 ? __syncthreads_or(__popcll(m_own) > 32) : 0;
        const int packed = block_sum((m_own != 0ull ? 1 : 0) + (__popcll(m_own) << 10), s_sum);
        const int nG = packed & 1023, npairs = packed >> 10;
        int nBig = 0;
#pragma unroll
        for (int i = 0; i < kMaxExperts / 64; ++i) nBig += __popcll(s_big[i]);
        const int tiles = (nG + nBig) * 8;
        if (tiles >= grid && tiles <= kTileSlots * grid) {
            tile_units_bits<GATED, kTileParts, true>(P, D, m_own, s_mask, s_kept, nG, stok,
                                                     reinterpret_cast<float4 *>(xf), s_big, nBig);
            return;
        }
        // Between half a tile and one tile per workgroup, past the small
        // unions: the same units in four parts (each wavefront a K quarter),
        // which keeps twice the wavefronts streaming
        if (nG > kSmallUnion && 2 * tiles >= grid && tiles < grid) {
            tile_units_bits<GATED, 2 * kTileParts, true>(P, D, m_own, s_mask, s_kept, nG, stok,
                                                         reinterpret_cast<float4 *>(xf), s_big, nBig);
            return;
        }
        // A small union (at most kSmallUnion kept experts, at most one tile
        // per workgroup): whole-workgroup tile units, eight K parts summed in
        // LDS -- as many bytes in flight per unit as a K-slice unit, without
        // the K-slice hand-off between workgroups
        if (!over32 && nG <= kSmallUnion && tiles <= grid && npairs <= 4 * nG) {
            float4 *red = reinterpret_cast<float4 *>(xf);
            if (GATED && nG >= kStreamGroups)
                tile_units_bits<GATED, kGuThreads / 64, true>(P, D, m_own, s_mask, s_kept, nG,
                                                              stok, red, s_big, 0);
            else
                tile_units_bits<GATED, kGuThreads / 64, false>(P, D, m_own, s_mask, s_kept, nG,
                                                               stok, red, s_big, 0);
            return;
        }
    }
    decode_plan<true>(P, D, m_own);
    const int nG = D.nG, npairs = D.npairs;
    // K-slices: KS per group, and one more for the first `extra` groups, so
    // that the units fill the resident workgroups exactly -- every CU then
    // streams the same number of units (with units left over, the CUs that
    // hold one unit fewer finish early and the rest form a tail)
    const int slots = (int)gridDim.x;
    const int KS = choose_ks(P, nG, npairs, slots);
    const int max_ks = max_slices(P, nG);
    int extra = 0;
    if (KS < max_ks && (size_t)(KS + 1) * npairs <= P.abpart_rows)
        extra = min(nG, max(0, slots - nG * KS));
    const int big = extra * (KS + 1);
    const int units = nG * KS + extra;
    // streaming weight loads for large unions (the K-slice units of non-gated
    // layers keep plain loads: their kernel for batches past 32 tokens has no
    // registers left for a second copy of the unit loop)
    const bool stream = GATED && __builtin_amdgcn_readfirstlane(nG) >= kStreamGroups;
    for (int unit = (int)blockIdx.x; unit < units; unit += slots) {
        int g, ks, ksg;
        if (unit < big) {
            g = unit / (KS + 1);
            ks = unit - g * (KS + 1);
            ksg = KS + 1;
        } else {
            const int v = unit - big;
            g = extra + v / KS;
            ks = v - (g - extra) * KS;
            ksg = KS;
        }
        const unsigned long long m = D.mask[g];
        if (tid < 64 && ((m >> tid) & 1ull)) stok[__popcll(m & ((1ull << tid) - 1ull))] = tid;
        __syncthreads();
        if (stream)
            gateup_group<GATED, NTMAX, PF, true>(P, D.e[g], __popcll(m), D.pair[g], g, ks, ksg,
                                                 npairs, stok, xf, &s_flag);
        else
            gateup_group<GATED, NTMAX, PF, false>(P, D.e[g], __popcll(m), D.pair[g], g, ks, ksg,
                                                  npairs, stok, xf, &s_flag);
        __syncthreads();
    }
}

// ------------------------------------------------------------------ down

// One (group, 16-token tile) of work in one 16-row tile of d, as held in
// registers by a wavefront: the tile's down fragments (4 K-steps of A) and
// the tokens' B fragments (h hi and lo).
template <int R>
struct RowItem {
    uint4 w[R][4];
    uint4 bh[4], bl[4];
    int tok;  // token of this lane's slot, -1 if the slot is empty
    bool live;
};

// Walks a wavefront's items: groups u = first, first + stride, ..., and the
// 16-token tiles of each group.
struct RowCursor {
    int u, j, n, p0, tk, e;
    int stride, nU;
    __device__ void enter(const PlanView &pl) {
        if (u < nU) {
            n = pl.grp_n[u];
            p0 = pl.grp_pair[u];
            tk = pl.grp_tok[u];
            e = pl.grp_e[u];
        }
    }
    __device__ void advance(const PlanView &pl) {
        if (16 * ++j >= n) {
            u += stride;
            j = 0;
            enter(pl);
        }
    }
};

template <int R, bool STREAM>
__device__ __forceinline__ void load_row_item(const DNParams &P, RowCursor &c, int rt, int RT,
                                              int lane, RowItem<R> &it) {
    const uint4 z = make_uint4(0, 0, 0, 0);
    it.live = c.u < c.nU;
    if (!it.live) return;
#pragma unroll
    for (int m = 0; m < R; ++m) {
        const uint16_t *wp = P.Wd + (((size_t)c.e * RT + rt + m) * 4 * 64 + lane) * 8;
#pragma unroll
        for (int s = 0; s < 4; ++s) it.w[m][s] = ldw16_if<STREAM>(wp + s * 512);
    }
    const int slot = 16 * c.j + (lane & 15);
    const bool ok = slot < c.n;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const size_t o = (size_t)(c.p0 + slot) * kExpertWidth + s * kKStep + 8 * (lane >> 4);
        it.bh[s] = ok ? ldg16(P.h_hi + o) : z;
        it.bl[s] = ok ? ldg16(P.h_lo + o) : z;
    }
    it.tok = ok ? P.plan.toklist[c.tk + slot] : -1;
    c.advance(P.plan);
}

// acc[t][16 R rows] += the item's 16 R x 16 block.
template <int R, int YS>
__device__ __forceinline__ void apply_row_item(const RowItem<R> &it, int lane, float (*acc)[YS]) {
#pragma unroll
    for (int m = 0; m < R; ++m) {
        f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            a = mfma16(it.w[m][s], it.bh[s], a);
            a = mfma16(it.w[m][s], it.bl[s], a);
        }
        // lane holds rows 4 (lane / 16) + i of tile m, token slot lane % 16
        if (it.tok >= 0) {
            float4 *dst = reinterpret_cast<float4 *>(&acc[it.tok][16 * m + 4 * (lane >> 4)]);
            float4 v = *dst;
            v.x += a[0];
            v.y += a[1];
            v.z += a[2];
            v.w += a[3];
            *dst = v;
        }
    }
}

// Unit = one 16-row tile of d over every group of the plan; wavefront w takes
// groups w, w + 8, ..., tile by tile of 16 tokens, with three tiles in
// flight, and adds into its own LDS accumulator [tokens][16 rows].  The eight accumulators are summed in
// wavefront order and the rows of y written once: no partial outputs, no
// cross-workgroup hand-off, every unit the same amount of work.
// ---- dense groups (many tokens per group): h shared through LDS

struct DnShared {
    float yacc[kDecodeTile][kShYS];
    uint4 hb[kShTiles][8][64];  // [token tile][hi s0..3, lo s0..3][lane]: B fragments
};
template <int TB, int R>
struct DnRow {
    float yacc[kDnThreads / 64][TB][16 * R + 4];
};

// This wavefront's 16 x 128 block of group u's down weights (row tile rt,
// clamped into d: a wavefront past d loads the last tile and discards it).
__device__ __forceinline__ void sh_load_w(const DNParams &P, int u, int rt, int RT, int lane,
                                          uint4 (&w)[4]) {
    const uint16_t *wp =
        P.Wd + (((size_t)P.plan.grp_e[u] * RT + min(rt, RT - 1)) * 4 * 64 + lane) * 8;
#pragma unroll
    for (int s = 0; s < 4; ++s) w[s] = ldw16(wp + s * 512);
}

// Piece wv (hi/lo x K-step) of group u's h B fragments and the tokens of
// this lane's slot, for every 16-token tile.  Bounds-checked buffer loads:
// every load is issued, slots past the group read zeros (their outputs are
// never stored), so the waits for a group's data count only later loads.
__device__ __forceinline__ void sh_load_h(const DNParams &P, int u, int wv, int lane,
                                          uint4 (&hp)[kShTiles], unsigned (&tp)[kShTiles]) {
    const int n = P.plan.grp_n[u], p0 = P.plan.grp_pair[u], tk = P.plan.grp_tok[u];
    const uint16_t *src = (__builtin_amdgcn_readfirstlane(wv) < 4) ? P.h_hi : P.h_lo;
    const auto rh = buf_rsrc(src + (size_t)p0 * kExpertWidth, (unsigned)n * kExpertWidth * 2u);
    const auto rt = buf_rsrc(P.plan.toklist + tk, (unsigned)n * 4u);
    const unsigned col = ((wv & 3) * kKStep + 8 * (lane >> 4)) * 2u;
#pragma unroll
    for (int j = 0; j < kShTiles; ++j) {
        const unsigned slot = 16 * j + (lane & 15);
        const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rh, slot * kExpertWidth * 2u + col, 0, 0);
        hp[j] = make_uint4(v.x, v.y, v.z, v.w);
        tp[j] = __builtin_amdgcn_raw_buffer_load_b32(rt, slot * 4u, 0, 0);
    }
}

// One group of a dense unit: stage its h in LDS, reuse hp for group u + 2's
// h, multiply, reuse wc for group u + 2's weights (both two groups ahead,
// clamped to the chunk's last group so that every group issues the same loads).
__device__ __forceinline__ void sh_group(const DNParams &P, DnShared &S, int u, int u1, int rt,
                                         int RT, bool rows_ok, int wv, int lane,
                                         uint4 (&hp)[kShTiles], unsigned (&tp)[kShTiles],
                                         uint4 (&wc)[4]) {
    const int n = P.plan.grp_n[u], nt = (n + 15) >> 4;
    unsigned tok[kShTiles];
    __syncthreads();  // every wavefront is done with the previous group's h
#pragma unroll
    for (int j = 0; j < kShTiles; ++j) {
        if (j < nt) S.hb[j][wv][lane] = hp[j];
        tok[j] = tp[j];
    }
    __syncthreads();
    const int un = min(u + 2, u1 - 1);
    sh_load_h(P, un, wv, lane, hp, tp);
    if (rows_ok) {
        for (int j = 0; j < nt; ++j) {
            f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                a = mfma16(wc[s], S.hb[j][s][lane], a);
                a = mfma16(wc[s], S.hb[j][4 + s][lane], a);
            }
            unsigned t = tok[0];
#pragma unroll
            for (int q = 1; q < kShTiles; ++q)
                if (j == q) t = tok[q];
            // lane holds rows 4 (lane / 16) + i of the wavefront's tile, token slot lane % 16
            if (16 * j + (lane & 15) < n) {
                float4 *dst = reinterpret_cast<float4 *>(&S.yacc[t][wv * 16 + 4 * (lane >> 4)]);
                float4 v = *dst;
                v.x += a[0];
                v.y += a[1];
                v.z += a[2];
                v.w += a[3];
                *dst = v;
            }
        }
    }
    sh_load_w(P, un, rt, RT, lane, wc);
}

// Dense unit = (chunk c of Uc groups, 128 rows of d): the 8 wavefronts own 16
// rows each and walk the chunk's groups together; the chunk's partial is
// summed with the other chunks' in chunk order by the last to arrive.
__device__ void sh_unit(const DNParams &P, DnShared &S, int c, int rb, int Uc, int nU, int ES,
                        int *flag) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int T = P.T, d = P.d, RT = d / 16;
    const int rt = rb * (kShRows / 16) + wv;
    const bool rows_ok = rt < RT;
    const int nrows = min(kShRows, d - rb * kShRows);
    for (int i = tid; i < T * kShYS; i += blockDim.x) S.yacc[i / kShYS][i % kShYS] = 0.0f;
    const int u0 = c * Uc, u1 = min(nU, u0 + Uc);
    uint4 w0[4], w1[4], hp0[kShTiles], hp1[kShTiles];
    unsigned tp0[kShTiles], tp1[kShTiles];
    const int u0n = min(u0 + 1, u1 - 1);
    sh_load_w(P, u0, rt, RT, lane, w0);
    sh_load_h(P, u0, wv, lane, hp0, tp0);
    sh_load_w(P, u0n, rt, RT, lane, w1);
    sh_load_h(P, u0n, wv, lane, hp1, tp1);
    for (int u = u0; u < u1; u += 2) {
        sh_group(P, S, u, u1, rt, RT, rows_ok, wv, lane, hp0, tp0, w0);
        if (u + 1 >= u1) break;
        sh_group(P, S, u + 1, u1, rt, RT, rows_ok, wv, lane, hp1, tp1, w1);
    }
    __syncthreads();
    const int nq = nrows / 4;
    const auto pr = buf_rsrc(P.ypart, (unsigned)((size_t)kDecodeChunks * T * d * 4u));
    for (int i = tid; i < T * nq; i += blockDim.x) {
        const int t = i / nq, r = 4 * (i - t * nq);
        float4 v = *reinterpret_cast<const float4 *>(&S.yacc[t][r]);
        const size_t col = (size_t)rb * kShRows + r;
        if (ES == 1) {
            if (P.bproj) {
                const float4 b = *reinterpret_cast<const float4 *>(P.bproj + col);
                v.x += b.x;
                v.y += b.y;
                v.z += b.z;
                v.w += b.w;
            }
            *reinterpret_cast<float4 *>(P.y + (size_t)t * d + col) = v;
        } else {
            st_dev16(pr, (unsigned)(((size_t)c * T + t) * d + col) * 4u, f32x4{v.x, v.y, v.z, v.w});
        }
    }
    if (ES == 1 || !arrive_last(&P.dn_cnt[rb], (unsigned)ES, flag)) return;
    // last chunk to arrive: y = sum of the chunk partials in chunk order, all
    // of a thread's 16-byte loads for kRedChunks chunks issued at once
    constexpr int kRedPer = kDecodeTile * (kShRows / 4) / kDnThreads;
    constexpr int kRedChunks = 4;
    const int nq4 = nrows / 4, nel = T * nq4;
    int off[kRedPer];
    f32x4 acc[kRedPer];
#pragma unroll
    for (int q = 0; q < kRedPer; ++q) {
        const int i = min(tid + kDnThreads * q, nel - 1), t = i / nq4;
        off[q] = t * d + rb * kShRows + 4 * (i - t * nq4);
        acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int nown = (nel - tid + kDnThreads - 1) / kDnThreads;
    for (int k0 = 0; k0 < ES; k0 += kRedChunks) {
        f32x4 v[kRedChunks][kRedPer];
#pragma unroll
        for (int k = 0; k < kRedChunks; ++k) {
            const size_t base = (size_t)min(k0 + k, ES - 1) * T * d;
#pragma unroll
            for (int q = 0; q < kRedPer; ++q)
                v[k][q] = q < nown ? ld_dev16(pr, (unsigned)(base + off[q]) * 4u)
                                   : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int k = 0; k < kRedChunks; ++k)
            if (k0 + k < ES)
#pragma unroll
                for (int q = 0; q < kRedPer; ++q) acc[q] += v[k][q];
    }
#pragma unroll
    for (int q = 0; q < kRedPer; ++q) {
        if (q < nown) {
            float4 o = make_float4(acc[q][0], acc[q][1], acc[q][2], acc[q][3]);
            if (P.bproj) {
                const float4 b = *reinterpret_cast<const float4 *>(P.bproj + off[q] % d);
                o.x += b.x;
                o.y += b.y;
                o.z += b.z;
                o.w += b.w;
            }
            *reinterpret_cast<float4 *>(P.y + off[q]) = o;
        }
    }
}

// Sparse groups: unit = R 16-row tiles of d over every group of the plan,
// the wavefronts' LDS accumulators summed in wavefront order and y written
// once.  STREAM: the down weights come by streaming (nontemporal) loads.
template <int TB, int R, bool STREAM>
__device__ void rows_sparse(const DNParams &P, DnRow<TB, R> &rw, int nU) {
    constexpr int YS = 16 * R + 4;
    constexpr int NW = kDnThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int RT = P.d / 16;
    float(*acc)[YS] = rw.yacc[wv];
    for (int rt = blockIdx.x * R; rt < RT; rt += gridDim.x * R) {
        for (int i = lane; i < P.T * YS; i += 64) acc[i / YS][i % YS] = 0.0f;
        RowCursor c;
        c.u = __builtin_amdgcn_readfirstlane(wv);
        c.j = 0;
        c.n = 0;
        c.stride = NW;
        c.nU = nU;
        c.enter(P.plan);
        // ring of kDnRing items: the next item's loads go out before each apply
        RowItem<R> it[kDnRing];
#pragma unroll
        for (int q = 0; q < kDnRing - 1; ++q) load_row_item<R, STREAM>(P, c, rt, RT, lane, it[q]);
        for (bool more = true; more;) {
#pragma unroll
            for (int q = 0; q < kDnRing; ++q) {
                if (!it[q].live) {
                    more = false;
                    break;
                }
                load_row_item<R, STREAM>(P, c, rt, RT, lane, it[(q + kDnRing - 1) % kDnRing]);
                apply_row_item<R, YS>(it[q], lane, acc);
            }
        }
        __syncthreads();
        for (int i = tid; i < P.T * 16 * R; i += blockDim.x) {
            const int t = i / (16 * R), r = i - t * 16 * R;
            float v = rw.yacc[0][t][r];
#pragma unroll
            for (int w = 1; w < NW; ++w) v += rw.yacc[w][t][r];
            if (P.bproj) v += P.bproj[rt * 16 + r];
            P.y[(size_t)t * P.d + rt * 16 + r] = v;
        }
        __syncthreads();
    }
}

template <int TB, int R>
__global__ __launch_bounds__(kDnThreads, 2) void down_dec_k(DNParams P) {
    __shared__ union {
        DnShared sh;
        DnRow<TB, R> rw;
    } S;
    __shared__ int s_flag;
    const int nU = P.plan.head[0], npairs = P.plan.head[1];
    // Dense groups (more than 16 tokens per group on average): reading h once
    // per 16-row tile would cost more than the weights, so share it through
    // LDS across 128-row units, with the groups split into chunks.  (Measured
    // crossover: at 6-16 tokens per group the row tiles are faster, at 28 the
    // shared h.)
    if (npairs > 16 * nU) {
        const int n_rb = (P.d + kShRows - 1) / kShRows;
        int ES = (int)gridDim.x / n_rb;
        if (ES > nU / 2) ES = nU / 2;
        if (ES > kDecodeChunks) ES = kDecodeChunks;
        if (ES < 1) ES = 1;
        const int Uc = (nU + ES - 1) / ES;
        ES = (nU + Uc - 1) / Uc;
        for (int unit = blockIdx.x; unit < ES * n_rb; unit += gridDim.x) {
            const int c = unit / n_rb, rb = unit - c * n_rb;
            sh_unit(P, S.sh, c, rb, Uc, nU, ES, &s_flag);
            __syncthreads();
        }
        return;
    }
    if (__builtin_amdgcn_readfirstlane(nU) >= kStreamGroups)
        rows_sparse<TB, R, true>(P, S.rw, nU);
    else
        rows_sparse<TB, R, false>(P, S.rw, nU);
}


// ---- every token keeps every expert (dense decode, up to 64 tokens): group u
// is expert u with all T tokens, its h rows u T .. u T + T - 1 in token order,
// so the outputs of a unit accumulate in registers across its groups with no
// per-group read-modify-write.  Unit = (32 NW rows of d, chunk of groups) on
// NW wavefronts; wavefront w owns row tiles 2 w and 2 w + 1 (each h fragment
// read from LDS feeds both).  Group u + 2's h fragments (copied into one of
// three LDS buffers by buffer loads to LDS) and weights (into a three-group
// register ring) are issued together at the start of group u, so every wait
// is for loads issued two groups earlier; one barrier per group.  The
// chunks store their partials and a second launch (dense_sum_k) sums them in
// chunk order on every CU.  Up to 32 tokens: four wavefronts (128 rows), two
// workgroups per CU; 64 tokens (three 32 KiB h buffers): eight wavefronts
// (256 rows), one workgroup per CU.
template <int NTT>
constexpr int dd_waves() { return NTT <= 2 ? 4 : 8; }

// Expert chunks of the dense kernel on `grid` workgroups over n_rb row
// blocks of nU groups: as many as fill the workgroups, at most nU / 3 (three
// groups per chunk) and kDecodeChunks; Uc groups per chunk.  The kernel and
// the host (which sizes the chunk sum) take it from here.
__host__ __device__ inline int dd_chunks(int grid, int nU, int n_rb, int *Uc) {
    int ES = grid / n_rb;
    if (ES > nU / 3) ES = nU / 3;
    if (ES > kDecodeChunks) ES = kDecodeChunks;
    if (ES < 1) ES = 1;
    *Uc = (nU + ES - 1) / ES;
    return (nU + *Uc - 1) / *Uc;
}

// Copies group u's h B fragments into hb: fragment f = (token tile f / 8,
// piece f % 8 = hi K-steps 0..3, lo K-steps 0..3); wavefront w of NW copies
// fragments w, w + NW, ...  Token slots past T read zeros.
template <int NTT>
__device__ __forceinline__ void dd_copy_h(const DNParams &P, uint4 (&hb)[NTT][8][64], int u,
                                          int wv, int lane) {
    constexpr int NW = dd_waves<NTT>();
    static_assert((8 * NTT) % NW == 0, "whole fragments per wavefront");
    const unsigned bytes = (unsigned)P.T * kExpertWidth * 2u;
    const size_t row0 = (size_t)u * P.T * kExpertWidth;
    const auto rh = buf_rsrc(P.h_hi + row0, bytes);
    const auto rl = buf_rsrc(P.h_lo + row0, bytes);
#pragma unroll
    for (int i = 0; i < 8 * NTT / NW; ++i) {
        const int f = wv + NW * i, j = f >> 3, pc = f & 7;
        const unsigned off =
            ((unsigned)(16 * j + (lane & 15)) * kExpertWidth + kKStep * (pc & 3) + 8 * (lane >> 4)) * 2u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            pc < 4 ? rh : rl, (__attribute__((address_space(3))) void *)&hb[j][pc][0], 16, off, 0, 0,
            0);
    }
}

// The wavefront's two row tiles of group u's down weights (row tiles past d
// load the last one and are discarded).  Every expert is kept, so group u is
// expert u (no plan load, whose wait would drain the loads in flight).
__device__ __forceinline__ void dd_load_w(const DNParams &P, int u, int rt0, int RT, int lane,
                                          uint4 (&w)[2][4]) {
    const int e = u;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const uint16_t *wp =
            P.Wd + (((size_t)e * RT + min(rt0 + t, RT - 1)) * 4 * 64 + lane) * 8;
#pragma unroll
        for (int s = 0; s < 4; ++s) w[t][s] = ldw16(wp + s * 512);
    }
}

// One group: wait for this wavefront's copies into cur (issued two groups
// ago), meet the other wavefronts (they are then done with group u - 1's
// buffer, which is nxt2), issue group u + 2's copies into nxt2 and weights
// into wl (group u - 1's ring slot), multiply cur with wu.
template <int NTT>
__device__ __forceinline__ void dd_group(const DNParams &P, const uint4 (&cur)[NTT][8][64],
                                         uint4 (&nxt2)[NTT][8][64], int u, int u1, int nt,
                                         int rt0, int RT, int wv, int lane, const uint4 (&wu)[2][4],
                                         uint4 (&wl)[2][4], f32x4 (&acc)[2][NTT]) {
    {
        // the last of this wavefront's copies into cur (fragment 8 NTT - NW + wv);
        // they complete in order
        constexpr int NW = dd_waves<NTT>();
        const int f = 8 * NTT - NW + wv;
        const uint4 own = cur[f >> 3][f & 7][lane];
        asm volatile("" ::"v"(own.x));
    }
    __syncthreads();
    // issued for every group (past the chunk: its last group again, into a
    // buffer and a ring slot no later group reads), so that the compiler's
    // waits count the same loads on every path
    const int un = min(u + 2, u1 - 1);
    dd_copy_h<NTT>(P, nxt2, un, wv, lane);
    dd_load_w(P, un, rt0, RT, lane, wl);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int j = 0; j < NTT; ++j) {
            if (j < nt) {
                const uint4 bh = cur[j][s][lane], bl = cur[j][4 + s][lane];
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    acc[t][j] = mfma16(wu[t][s], bh, acc[t][j]);
                    acc[t][j] = mfma16(wu[t][s], bl, acc[t][j]);
                }
            }
        }
    }
}

// NTT: token tiles the kernel holds (T <= 16 NTT).
template <int NTT>
__global__ __launch_bounds__(64 * dd_waves<NTT>(), 8 / dd_waves<NTT>()) void down_dense_k(DNParams P) {
    constexpr int kDdThreads = 64 * dd_waves<NTT>();
    constexpr int kDdRows = 32 * dd_waves<NTT>();
    __shared__ uint4 hb0[NTT][8][64];
    __shared__ uint4 hb1[NTT][8][64];
    __shared__ uint4 hb2[NTT][8][64];
    // the wavefront index in a scalar register: the copies' descriptors and LDS
    // addresses derive from it and must be known uniform
    const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int T = P.T, d = P.d, RT = d / 16, nt = (T + 15) >> 4;
    const int nU = P.E;  // every expert is a group
    const int n_rb = (d + kDdRows - 1) / kDdRows;
    int Uc;
    const int ES = dd_chunks((int)gridDim.x, nU, n_rb, &Uc);
    const auto pr = buf_rsrc(P.ypart, (unsigned)((size_t)kDecodeChunks * T * d * 4u));
    for (int unit = blockIdx.x; unit < ES * n_rb; unit += gridDim.x) {
        const int c = unit / n_rb, rb = unit - c * n_rb;
        const int rt0 = rb * (kDdRows / 16) + 2 * wv;
        const int u0 = c * Uc, u1 = min(nU, u0 + Uc);
        f32x4 acc[2][NTT];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int j = 0; j < NTT; ++j) acc[t][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        uint4 w0[2][4], w1[2][4], w2[2][4];
        dd_copy_h<NTT>(P, hb0, u0, wv, lane);
        dd_load_w(P, u0, rt0, RT, lane, w0);
        dd_copy_h<NTT>(P, hb1, min(u0 + 1, u1 - 1), wv, lane);
        dd_load_w(P, min(u0 + 1, u1 - 1), rt0, RT, lane, w1);
        for (int u = u0; u < u1; u += 3) {
            dd_group<NTT>(P, hb0, hb2, u, u1, nt, rt0, RT, wv, lane, w0, w2, acc);
            if (u + 1 >= u1) break;
            dd_group<NTT>(P, hb1, hb0, u + 1, u1, nt, rt0, RT, wv, lane, w1, w0, acc);
            if (u + 2 >= u1) break;
            dd_group<NTT>(P, hb2, hb1, u + 2, u1, nt, rt0, RT, wv, lane, w2, w1, acc);
        }
        // lane holds rows 4 (lane / 16) + i of row tile rt0 + t, token slot 16 j + lane % 16
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int j = 0; j < NTT; ++j) {
                const int tok = 16 * j + (lane & 15);
                if (rt0 + t < RT && tok < T) {
                    const int col = (rt0 + t) * 16 + 4 * (lane >> 4);
                    f32x4 v = acc[t][j];
                    if (ES == 1) {
                        if (P.bproj) v += *reinterpret_cast<const f32x4 *>(P.bproj + col);
                        *reinterpret_cast<f32x4 *>(P.y + (size_t)tok * d + col) = v;
                    } else {
                        // the sum runs in the next launch, so a plain store is
                        // enough; the 64-token build measured faster with it
                        // (100.7 vs 102.2 us per step), the smaller ones with
                        // the device-coherent store (89.4 vs 89.9 us at T = 32)
                        const unsigned o = (unsigned)(((size_t)c * T + tok) * d + col) * 4u;
                        if (NTT > 2)
                            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), pr, o, 0, 0);
                        else
                            st_dev16(pr, o, v);
                    }
                }
            }
        }
        __syncthreads();  // the unit's LDS buffers are free again
    }
}

// y of a dense batch split into ES expert chunks: y = sum of the chunk
// partials in chunk order (+ the output bias), one 16-byte piece per thread,
// all of its ES loads in flight at once.  A launch of its own after the
// chunks: every CU sums, where the last chunk to arrive of a row block
// summed its whole block alone (the kernel's tail).
__global__ __launch_bounds__(256) void dense_sum_k(DNParams P, int ES) {
    const int n4 = P.T * (P.d / 4);
    const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (i >= n4) return;
    const size_t off = (size_t)i * 4, slab = (size_t)P.T * P.d;
    f32x4 v[kDecodeChunks];
#pragma unroll
    for (int k = 0; k < kDecodeChunks; ++k)
        v[k] = *reinterpret_cast<const f32x4 *>(P.ypart + (size_t)min(k, ES - 1) * slab + off);
    f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < kDecodeChunks; ++k)
        if (k < ES) a += v[k];
    if (P.bproj) a += *reinterpret_cast<const f32x4 *>(P.bproj + off % P.d);
    *reinterpret_cast<f32x4 *>(P.y + off) = a;
}

template <int NTT>
void launch_down_dense(const DNParams &dp, int num_cu, hipStream_t s) {
    constexpr int threads = 64 * dd_waves<NTT>(), rows = 32 * dd_waves<NTT>();
    static const int occ = resident(down_dense_k<NTT>, threads);
    const int grid = occ * num_cu;
    hipLaunchKernelGGL(down_dense_k<NTT>, dim3(grid), dim3(threads), 0, s, dp);
    int Uc;
    const int ES = dd_chunks(grid, dp.E, (dp.d + rows - 1) / rows, &Uc);
    if (ES > 1) {
        const int n4 = dp.T * (dp.d / 4);
        hipLaunchKernelGGL(dense_sum_k, dim3((n4 + 255) / 256), dim3(256), 0, s, dp, ES);
    }
}

// ------------------------------------------------------------------ launchers

template <int TB>
void launch_down_dec_tb(const DNParams &P, int num_cu, hipStream_t s) {
    constexpr int R = kDnR;
    static const int occ = resident(down_dec_k<TB, R>, kDnThreads);
    const int units = P.d / (16 * R);
    const int grid = units < occ * num_cu ? units : occ * num_cu;
    hipLaunchKernelGGL((down_dec_k<TB, R>), dim3(grid), dim3(kDnThreads), 0, s, P);
}

}  // namespace

// gate/up of a decode slice of T tokens: groups hold at most T tokens, so
// the kernel is compiled for at most ceil(T / 16) token tiles, and the
// registers the larger tiles would take go to a deeper weight prefetch.
template <bool GATED, int NTMAX, int PF>
void launch_gateup_dec(const GUParams &gp, int num_cu, hipStream_t s) {
    static const int occ = resident(gateup_dec_k<GATED, NTMAX, PF>, kGuThreads);
    hipLaunchKernelGGL((gateup_dec_k<GATED, NTMAX, PF>), dim3(occ * num_cu), dim3(kGuThreads), 0, s,
                       gp);
}

template <bool GATED>
void launch_gateup_dec_t(const GUParams &gp, int T, int num_cu, hipStream_t s) {
    if (T <= 16)
        launch_gateup_dec<GATED, 1, 3>(gp, num_cu, s);
    else if (T <= 32)
        launch_gateup_dec<GATED, 2, 3>(gp, num_cu, s);
    else
        launch_gateup_dec<GATED, 4, kPF>(gp, num_cu, s);
}

hipError_t launch_decode_ffn(pp_layer *L, const uint16_t *x, int T, float *y, bool dense,
                             hipStream_t s, const DecodeSelect *sel) {
    GUParams gp = gu_params(L, x, T, false);
    if (sel) {
        if (T != 1 || dense) return hipErrorInvalidValue;
        gp.select_here = 1;
        gp.rp = route_params(L, x, T, sel->tau, sel->inv_temp, sel->idx, sel->count, nullptr,
                             false);
    }
    prof_mark(L, PP_KERNEL_GATEUP, s, true);
    // dense batches of more than 24 tokens: the grouped kernel, which stages
    // the tokens in LDS once per group; up to 24 tokens the neuron-tile units
    // (tokens read from x per unit) stream faster (T = 16 / 24, tau 1: 49.6 /
    // 51.3 -> 42.9 / 47.6 us; at 32 tokens 51.5 -> 57.4 us)
    if (dense && T > 24)
        launch_gateup_dense_dec(L, x, T, s);
    else if (L->gated)
        launch_gateup_dec_t<true>(gp, T, L->num_cu, s);
    else
        launch_gateup_dec_t<false>(gp, T, L->num_cu, s);
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
    dp.bproj = L->bproj;
    dp.ypart = L->ypart;
    dp.dn_cnt = L->counters + counters_for(L->dm, L->max_tokens).down_base();
    dp.plan = plan_view(L, false);
    prof_mark(L, PP_KERNEL_DOWN, s, true);
    if (dense && T <= 16)
        launch_down_dense<1>(dp, L->num_cu, s);
    else if (dense && T <= 32)
        launch_down_dense<2>(dp, L->num_cu, s);
    else if (dense)
        launch_down_dense<4>(dp, L->num_cu, s);
    else if (T <= 16)
        launch_down_dec_tb<16>(dp, L->num_cu, s);
    else if (T <= 32)
        launch_down_dec_tb<32>(dp, L->num_cu, s);
    else
        launch_down_dec_tb<64>(dp, L->num_cu, s);
    prof_mark(L, PP_KERNEL_DOWN, s, false);
    return hipGetLastError();
}

}  // namespace pp
