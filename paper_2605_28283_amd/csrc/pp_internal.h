// Internal declarations of the gfx950 PrunePath library: the layer handle,
// kernel parameter blocks, launchers and small device helpers shared by the
// kernel files.  Nothing here is part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/prunepath.h"

namespace pp {

constexpr int kExpertWidth = 128;      // neurons per expert (de)
constexpr int kKStep = 32;             // K per bf16 MFMA 16x16x32
constexpr int kMaxExperts = 256;
constexpr int kDecodeTile = 64;        // tokens per decode slice (one u64 token mask)
constexpr int kDecodeChunks = 16;      // expert chunks of the dense-group decode down projection
constexpr int kRouteTile = 16;         // tokens / experts per router MFMA tile
constexpr int kMaxWidth = 8192;        // largest supported d
constexpr int kPfChunk = 512;          // tokens per prefill down unit (their y rows stay in LDS)
constexpr int kGroupTokens = 64;       // tokens per decode expert group (one u64 token mask)
constexpr int kPfGroupTokens = 128;    // tokens per prefill expert group
constexpr int kMinStepsPerSlice = 8;   // K-steps each gate/up K-slice covers at least
constexpr int kMaxSlicesSmallUnion = 8;  // K-slices per group when at most kSmallUnion experts are kept
constexpr int kSmallUnion = 32;

// Byte sizes of the scratch areas whose size does not follow from max_tokens.
constexpr size_t kAbPartRows = 65536;  // K-split partial (a,b) rows of 256 floats

struct pp_dims {
    int d, d_ff, E, NS;      // NS = d / 32 K-steps
};

struct profiler;  // per-kernel event timing (benchmarking aid)

// Work plan of one FFN call (device memory): head[0] = number of groups,
// head[1] = number of (token, expert) pair rows; group g is expert grp_e[g]
// with grp_n[g] <= 64 tokens toklist[grp_tok[g] .. + grp_n[g]) whose h rows
// start at grp_pair[g].
struct PlanView {
    int32_t *head;
    int32_t *grp_e;
    int32_t *grp_pair;
    int32_t *grp_n;
    int32_t *grp_tok;
    int32_t *toklist;
    int32_t *egrp;  // prefill: expert e owns groups [egrp[e], egrp[e + 1])
};

// Work-unit order for persistent grids whose size is a multiple of 8: the
// workgroups of one XCD (blockIdx % 8 on MI355X's eight XCDs) take one
// contiguous range of unit indices, so neighbouring units -- which share
// inputs, e.g. one expert's weights or h rows -- meet in the same L2.
// Returns the unit that linear slot `u` of `n` stands for.
__host__ __device__ inline int xcd_order(int u, int n) {
    const int per = (n + 7) / 8;
    return (u % 8) * per + u / 8;
}

// Largest number of groups a call can produce.
inline int plan_max_groups(const pp_dims &dm, int max_tokens) {
    return dm.E + (int)(((long)max_tokens * dm.E + 63) / 64);
}

// Brackets one kernel launch with profiling events when the handle records.
void prof_mark(pp_layer *L, int kind, hipStream_t s, bool start);

}  // namespace pp

struct pp_layer {
    pp::pp_dims dm;
    int max_tokens;
    uint32_t flags;
    bool gated;        // SwiGLU (true) or the non-gated GELU MLP with biases
    int device;
    int num_cu;
    // library-owned weights
    uint16_t *Wr;      // [E][d] bf16
    float *bias;       // [E] fp32 (zeros when the caller gave none)
    uint16_t *Wgu;     // expert-major gate/up (or W_fc) MFMA fragments
    uint16_t *Wd;      // expert-major down (or W_proj) MFMA fragments
    float *bfc;        // non-gated: [d_ff] input bias in expert order (Pi applied)
    float *bproj;      // non-gated: [d] output bias, or NULL
    // scratch
    float *gpart;       // router K-slice partial logits [d/512][max_tokens][E]
    size_t gpart_elems;
    uint32_t *counters; // arrival counters, zero between calls
    size_t n_counters;
    uint32_t *selmask;  // [max_tokens][8] kept-expert bitmask per token
    float *gsig;        // [max_tokens][E] expert scale (sigmoid(g) or 1)
    int32_t *idx_tmp;   // [max_tokens][E] used when the caller passes no expert_idx
    int32_t *cnt_tmp;   // [max_tokens]
    float *abpart;      // [kAbPartRows][256] K-split partial gate/up outputs
    uint16_t *h_hi;     // [pairs][128] bf16 high part of h
    uint16_t *h_lo;     // [pairs][128] bf16 low part of h (h - hi)
    size_t max_pairs;
    float *ypart;       // [kDecodeChunks][kDecodeTile][d] chunk partial outputs (decode, dense groups)
    int32_t *ecount;    // [E] tokens per expert (prefill)
    int32_t *tokl;      // [E][max_tokens] token ids per expert (prefill)
    int32_t *pf_cut;    // prefill: [E][pf_ncut] bucket position where each token chunk starts
    int pf_ncut;        // token chunks of the largest batch + 1
    int32_t *pf_ebase;  // prefill: [E] first pair row of each expert's bucket
    int32_t *plan;      // PlanView storage: 4 + 4 * plan_max_groups + E + 1 ints
    int32_t *dec_tok;   // [64 * E] token ids of the decode plan, pair order
    unsigned long long *emask;  // [E] decode: tokens that kept each expert (zero between calls)
    pp::profiler *prof; // non-NULL while per-kernel timing is recorded
};

namespace pp {

// Counter regions inside pp_layer::counters (all zero at create; every
// arrival counter is reset by its last arriver).
struct counter_layout {
    size_t route;     // none
    size_t gateup;    // one per group: K-slice arrivals
    size_t down;      // one per 128-row block: decode chunk arrivals
    size_t dispatch;  // one: prefill bucketing arrivals
    size_t total;
    size_t gateup_base() const { return route; }
    size_t down_base() const { return route + gateup; }
    size_t dispatch_base() const { return route + gateup + down; }
};
counter_layout counters_for(const pp_dims &dm, int max_tokens);

inline PlanView plan_view(pp_layer *L, bool prefill);


// W_up NULL: non-gated layer (one input projection per expert); b_fc, if
// given, is copied into expert order.
hipError_t launch_repack(pp_layer *L, const uint16_t *W_gate, const uint16_t *W_up,
                         const uint16_t *W_down, const int32_t *perm, const float *b_fc,
                         hipStream_t s);
// select = false launches the router logits only (the single-token decode
// gate/up kernel then selects the token's experts itself).
hipError_t launch_route(pp_layer *L, const uint16_t *x, int T, float tau, const float *inv_temp,
                        int32_t *idx, int32_t *count, float *gate_w, bool build_plan,
                        hipStream_t s, bool select = true);
// dense: every token keeps every expert (the gate/up then runs as grouped
// MFMA work like prefill).
// The selection arguments of a single-token decode call whose gate/up
// kernel selects the experts itself (after launch_route with select = false).
struct DecodeSelect {
    float tau;
    const float *inv_temp;
    int32_t *idx;
    int32_t *count;
};
hipError_t launch_decode_ffn(pp_layer *L, const uint16_t *x, int T, float *y, bool dense,
                             hipStream_t s, const DecodeSelect *sel = nullptr);
void launch_gateup_dense_dec(pp_layer *L, const uint16_t *x, int T, hipStream_t s);
hipError_t launch_prefill_ffn(pp_layer *L, const uint16_t *x, int T, float *y, hipStream_t s);

inline PlanView plan_view(pp_layer *L, bool prefill) {
    const int G = plan_max_groups(L->dm, L->max_tokens);
    PlanView v;
    v.head = L->plan;
    v.grp_e = L->plan + 4;
    v.grp_pair = v.grp_e + G;
    v.grp_n = v.grp_pair + G;
    v.grp_tok = v.grp_n + G;
    v.toklist = prefill ? L->tokl : L->dec_tok;
    v.egrp = v.grp_tok + G;
    return v;
}

// ---------------------------------------------------------------- device helpers
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x4 mfma16(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__device__ __forceinline__ uint4 ldg16(const void *p) {
    return *reinterpret_cast<const uint4 *>(p);
}

// A weight fragment read once per call: a nontemporal load (streamed past the
// caches).  When a call touches only a few experts, their weights can stay in
// the Infinity Cache between calls, so plain loads are kept for small unions
// (fewer than kStreamGroups kept experts, decided per call on the device).
__device__ __forceinline__ uint4 ldw16(const void *p) {
    typedef unsigned int v4 __attribute__((ext_vector_type(4)));
    const v4 v = __builtin_nontemporal_load(reinterpret_cast<const v4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
template <bool STREAM>
__device__ __forceinline__ uint4 ldw16_if(const void *p) {
    return STREAM ? ldw16(p) : ldg16(p);
}
constexpr int kStreamGroups = 16;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// A raw buffer over [base, base + bytes): loads past it read zeros without a
// memory access, so a load can be issued whether or not its lane has data.
// base and bytes must be wavefront-uniform; they are moved to scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *base, unsigned bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    const uint32_t nb = __builtin_amdgcn_readfirstlane(bytes);
    return __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void *>(((uint64_t)hi << 32) | lo), (short)0, (int)nb, 0x00020000);
}

__device__ __forceinline__ float silu(float a) { return a / (1.0f + expf(-a)); }

// ------------------------------------------------ hand-off between workgroups
// Partial results that one workgroup passes to another inside the same kernel
// are written and read with agent-scope relaxed atomic accesses, which gfx950
// performs at the device coherence point (the per-XCD L2s are not coherent
// with each other).  The writer waits for its stores to complete before it
// bumps the arrival counter; the last arriver then reads with the same scope.
// No cache-wide writeback or invalidate is needed, so other workgroups keep
// their L2 contents.
__device__ __forceinline__ void st_dev(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev2(float *p, float a, float b) {
    const unsigned long long u =
        (unsigned long long)__float_as_uint(a) | ((unsigned long long)__float_as_uint(b) << 32);
    __hip_atomic_store(reinterpret_cast<unsigned long long *>(p), u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev_u32(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_dev_u32(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_dev2(const float *p) {
    const unsigned long long u = __hip_atomic_load(
        reinterpret_cast<const unsigned long long *>(p), __ATOMIC_RELAXED,
        __HIP_MEMORY_SCOPE_AGENT);
    return make_float2(__uint_as_float((uint32_t)u), __uint_as_float((uint32_t)(u >> 32)));
}
// 16-byte stores and loads at the device coherence point through a raw
// buffer (cache policy sc1, what the agent-scope atomic stores and loads
// above compile to), for partial results laid out in MFMA fragment order:
// one wavefront instruction then moves one contiguous KiB instead of
// scattered 8-byte pieces.
constexpr int kCpolDevice = 16;  // sc1
__device__ __forceinline__ void st_dev16(__amdgpu_buffer_rsrc_t r, unsigned off, f32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, off, 0, kCpolDevice);
}
__device__ __forceinline__ f32x4 ld_dev16(__amdgpu_buffer_rsrc_t r, unsigned off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCpolDevice));
}

// Wait until this thread's outstanding vector-memory operations completed
// (s_waitcnt vmcnt(0); the expcnt and lgkmcnt fields are left at their maxima).
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Arrival on a counter shared by `n` workgroups after each has stored its
// partial results with st_dev*; returns true in exactly one workgroup, the
// last to arrive, which also resets the counter for the next call.  Must be
// reached by every thread of the workgroup.  `flag` is a shared int.
__device__ __forceinline__ bool arrive_last(uint32_t *counter, unsigned n, int *flag) {
    wait_vmem();
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned old =
            __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int last = (old == n - 1u);
        if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *flag = last;
    }
    __syncthreads();
    return *flag != 0;
}

// ------------------------------------------------ cross-lane exchange (no LDS)
// Value of lane (lane ^ ST) for ST = 1..32, built from DPP row operations
// (quad permutes, row shifts, row rotate) and the gfx950 permlane swaps.
template <int ST>
__device__ __forceinline__ uint32_t xor_lane(uint32_t v, int lane) {
    if constexpr (ST == 1) {
        return __builtin_amdgcn_update_dpp(0u, v, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
    } else if constexpr (ST == 2) {
        return __builtin_amdgcn_update_dpp(0u, v, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
    } else if constexpr (ST == 4) {
        const uint32_t up = __builtin_amdgcn_update_dpp(0u, v, 0x104, 0xF, 0xF, false);  // i <- i+4
        const uint32_t dn = __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xF, 0xF, false);  // i <- i-4
        return (lane & 4) ? dn : up;
    } else if constexpr (ST == 8) {
        return __builtin_amdgcn_update_dpp(0u, v, 0x128, 0xF, 0xF, false);  // row_ror:8
    } else if constexpr (ST == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return (lane & 16) ? r[0] : r[1];
    } else {
        static_assert(ST == 32, "xor_lane: stride must be a power of two below 64");
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return (lane & 32) ? r[0] : r[1];
    }
}

__device__ __forceinline__ uint32_t xor_lane_rt(uint32_t v, int st, int lane) {
    switch (st) {
    case 1: return xor_lane<1>(v, lane);
    case 2: return xor_lane<2>(v, lane);
    case 4: return xor_lane<4>(v, lane);
    case 8: return xor_lane<8>(v, lane);
    case 16: return xor_lane<16>(v, lane);
    default: return xor_lane<32>(v, lane);
    }
}

// Inclusive prefix sum of one float per lane over the 64-lane wavefront, in
// DPP row shifts (within rows of 16) and row broadcasts (across rows).
__device__ __forceinline__ float wave_scan_f32(float x) {
    x += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x111, 0xF, 0xF, false));
    x += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x112, 0xF, 0xF, false));
    x += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x114, 0xF, 0xF, false));
    x += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x118, 0xF, 0xF, false));
    x += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x142, 0xA, 0xF, false));
    x += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x143, 0xC, 0xF, false));
    return x;
}

// The same DPP prefix sum for one int per lane.
__device__ __forceinline__ int wave_scan_i32(int x) {
    x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x111, 0xF, 0xF, false);
    x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x112, 0xF, 0xF, false);
    x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x114, 0xF, 0xF, false);
    x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x118, 0xF, 0xF, false);
    x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x142, 0xA, 0xF, false);
    x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x143, 0xC, 0xF, false);
    return x;
}

__device__ __forceinline__ float lane_value(float x, int lane) {
    return __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), lane));
}

// Inclusive scan of one int per lane across a 64-lane wavefront.
__device__ __forceinline__ int wave_incl_scan(int v) { return wave_scan_i32(v); }

// Exclusive scan over a block of nthreads (multiple of 64, <= 1024) for two
// ints at once.  `sm` needs 2 * (nthreads/64) ints of shared memory.  Returns
// the exclusive prefixes; totals are written to *tot0 / *tot1 for every thread.
__device__ __forceinline__ void block_excl_scan2(int v0, int v1, int *e0, int *e1, int *tot0,
                                                 int *tot1, int *sm) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int i0 = wave_incl_scan(v0), i1 = wave_incl_scan(v1);
    if (lane == 63) {
        sm[wv] = i0;
        sm[nw + wv] = i1;
    }
    __syncthreads();
    int b0 = 0, b1 = 0, t0 = 0, t1 = 0;
#pragma unroll
    for (int w = 0; w < 16; ++w) {
        if (w < nw) {  // uniform: all of the wavefront totals are read at once
            const int a = sm[w], c = sm[nw + w];
            b0 += w < wv ? a : 0;
            b1 += w < wv ? c : 0;
            t0 += a;
            t1 += c;
        }
    }
    *e0 = b0 + i0 - v0;
    *e1 = b1 + i1 - v1;
    *tot0 = t0;
    *tot1 = t1;
    __syncthreads();
}

}  // namespace pp
