// C ABI entry points (include/prunepath.h): argument validation, ownership of
// the repacked weights and scratch, and the launch sequence of each call on
// the caller's stream.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "pp_internal.h"

namespace pp {

struct profiler {
    std::vector<hipEvent_t> ev;  // start/stop pairs
    std::vector<int> kind;
    int cap = 0, used = 0;
};

void prof_mark(pp_layer *L, int kind, hipStream_t s, bool start) {
    profiler *P = L->prof;
    if (!P || P->used >= P->cap) return;
    if (start) {
        (void)hipEventRecord(P->ev[2 * P->used], s);
        P->kind[P->used] = kind;
    } else {
        (void)hipEventRecord(P->ev[2 * P->used + 1], s);
        ++P->used;
    }
}

}  // namespace pp

namespace {

using namespace pp;

void free_profiler(profiler *P) {
    if (!P) return;
    for (hipEvent_t e : P->ev)
        if (e) (void)hipEventDestroy(e);
    delete P;
}

constexpr int kMaxTokensLimit = 65536;

template <typename T>
hipError_t dev_alloc(T **p, size_t elems) {
    *p = nullptr;
    if (elems == 0) elems = 1;
    return hipMalloc(reinterpret_cast<void **>(p), elems * sizeof(T));
}

void free_layer(pp_layer *L) {
    if (!L) return;
    void *bufs[] = {L->Wr,     L->bias,  L->Wgu,     L->Wd,    L->bfc,   L->bproj, L->gpart, L->counters,
                    L->selmask, L->gsig, L->idx_tmp, L->cnt_tmp, L->abpart, L->h_hi,
                    L->h_lo,   L->ypart, L->ecount,  L->tokl,  L->plan,  L->dec_tok,
                    L->pf_cut, L->pf_ebase,
                    L->emask};
    for (void *b : bufs)
        if (b) (void)hipFree(b);
    free_profiler(L->prof);
    delete L;
}

bool valid_tau(float tau) { return !isnan(tau) && tau >= 0.0f; }

pp_status check_call(const pp_layer *L, const uint16_t *x, int32_t T, float tau) {
    if (!L || !x) return PP_EINVAL;
    if (T < 1 || T > L->max_tokens) return PP_EINVAL;
    if (!valid_tau(tau)) return PP_EINVAL;
    return PP_OK;
}

pp_status hip_status(hipError_t e) {
    if (e == hipSuccess) return PP_OK;
    if (e == hipErrorOutOfMemory) return PP_ENOMEM;
    return PP_EHIP;
}

pp_status run_ffn(pp_layer *L, const uint16_t *x, int32_t T, float tau, const float *inv_temp,
                  float *y, int32_t *expert_idx, int32_t *count, void *hip_stream, bool prefill) {
    pp_status st = check_call(L, x, T, tau);
    if (st != PP_OK) return st;
    if (!y || ((expert_idx == nullptr) != (count == nullptr))) return PP_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    const int E = L->dm.E, d = L->dm.d;
    const int slice = prefill ? T : kDecodeTile;
    // every token keeps every expert (nucleus with tau >= 1, strict with
    // tau > 1, top-k with k >= E): a decode slice of at least 16 tokens then
    // runs its gate/up as grouped work (below 16 the K-split units are faster)
    const uint32_t sel = L->flags & (PP_SELECT_STRICT | PP_SELECT_TOPK | PP_SELECT_LTE);
    const bool all_kept = (sel == PP_SELECT_NUCLEUS && tau >= 1.0f) ||
                          (sel == PP_SELECT_STRICT && tau > 1.0f) ||
                          (sel == PP_SELECT_TOPK && floorf(tau + 0.5f) >= (float)E);
    for (int t0 = 0; t0 < T; t0 += slice) {
        const int n = (T - t0 < slice) ? T - t0 : slice;
        int32_t *idx = expert_idx ? expert_idx + (size_t)t0 * E : L->idx_tmp;
        int32_t *cnt = count ? count + t0 : L->cnt_tmp;
        const uint16_t *xs = x + (size_t)t0 * d;
        float *ys = y + (size_t)t0 * d;
        const float *it = inv_temp ? inv_temp + t0 : nullptr;
        // a single decode token: the gate/up kernel selects its experts itself
        // (one launch and one round trip fewer)
        const bool fuse = !prefill && n == 1;
        const DecodeSelect dsel = {tau, it, idx, cnt};
        hipError_t e = launch_route(L, xs, n, tau, it, idx, cnt, nullptr, !prefill && !fuse, s,
                                    !fuse);
        if (e == hipSuccess)
            e = prefill ? launch_prefill_ffn(L, xs, n, ys, s)
                        : launch_decode_ffn(L, xs, n, ys, all_kept && n >= 16, s,
                                            fuse ? &dsel : nullptr);
        if (e != hipSuccess) return hip_status(e);
    }
    return PP_OK;
}

}  // namespace

namespace {

// Both layer kinds: W_up NULL makes a non-gated layer (W_gate = W_fc,
// W_down = W_proj, optional biases b_fc and b_proj).
pp_status create_layer(pp_layer **out, int32_t d, int32_t d_ff, int32_t E, int32_t max_tokens,
                       const uint16_t *W_r, const uint16_t *W_gate, const uint16_t *W_up,
                       const uint16_t *W_down, const float *b_fc, const float *b_proj,
                       const int32_t *perm, const float *router_bias, uint32_t flags,
                       void *hip_stream) {
    const bool gated = W_up != nullptr;
    if (d < 1 || d_ff < 1 || E < 1 || max_tokens < 1 || max_tokens > kMaxTokensLimit)
        return PP_EINVAL;
    if (flags & ~(PP_SELECT_STRICT | PP_SELECT_TOPK | PP_SELECT_LTE | PP_AGG_SIGMOID))
        return PP_EINVAL;
    {
        const uint32_t sel = flags & (PP_SELECT_STRICT | PP_SELECT_TOPK | PP_SELECT_LTE);
        if (sel & (sel - 1u)) return PP_EINVAL;  // more than one selection rule
    }
    if (d_ff % E != 0) return PP_EINVAL;
    if (E > kMaxExperts) return PP_EUNSUPPORTED;
    if (d_ff / E != kExpertWidth) return PP_EUNSUPPORTED;
    if (d % 64 != 0 || d > kMaxWidth) return PP_EUNSUPPORTED;

    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    if (perm) {
        std::vector<int32_t> hp((size_t)d_ff);
        if (hipMemcpy(hp.data(), perm, sizeof(int32_t) * d_ff, hipMemcpyDeviceToHost) !=
            hipSuccess)
            return PP_EHIP;
        std::vector<unsigned char> seen((size_t)d_ff, 0);
        for (int32_t v : hp) {
            if (v < 0 || v >= d_ff || seen[v]) return PP_EINVAL;
            seen[v] = 1;
        }
    }

    pp_layer *L = new (std::nothrow) pp_layer;
    if (!L) return PP_ENOMEM;
    memset(L, 0, sizeof *L);
    L->dm.d = d;
    L->dm.d_ff = d_ff;
    L->dm.E = E;
    L->dm.NS = d / kKStep;
    L->max_tokens = max_tokens;
    L->flags = flags;
    L->gated = gated;
    hipError_t e = hipGetDevice(&L->device);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&L->num_cu, hipDeviceAttributeMultiprocessorCount, L->device);
    if (e != hipSuccess) {
        free_layer(L);
        return PP_EHIP;
    }

    const size_t dE = (size_t)d * E;
    const counter_layout cl = counters_for(L->dm, max_tokens);
    L->gpart_elems = (size_t)((L->dm.NS + 15) / 16) * max_tokens * E;
    L->n_counters = cl.total;
    L->max_pairs = (size_t)max_tokens * E;

    hipError_t a = hipSuccess;
    auto chk = [&](hipError_t r) {
        if (a == hipSuccess) a = r;
    };
    chk(dev_alloc(&L->Wr, dE));
    chk(dev_alloc(&L->bias, (size_t)E));
    chk(dev_alloc(&L->Wgu, (size_t)(gated ? 2 : 1) * d_ff * d));
    chk(dev_alloc(&L->Wd, (size_t)d_ff * d));
    if (!gated) {
        chk(dev_alloc(&L->bfc, (size_t)d_ff));
        if (b_proj) chk(dev_alloc(&L->bproj, (size_t)d));
    }
    chk(dev_alloc(&L->gpart, L->gpart_elems));
    chk(dev_alloc(&L->counters, L->n_counters));
    chk(dev_alloc(&L->selmask, (size_t)max_tokens * 8));
    chk(dev_alloc(&L->gsig, (size_t)max_tokens * E));
    chk(dev_alloc(&L->idx_tmp, (size_t)max_tokens * E));
    chk(dev_alloc(&L->cnt_tmp, (size_t)max_tokens));
    chk(dev_alloc(&L->abpart, kAbPartRows * 256));
    chk(dev_alloc(&L->h_hi, L->max_pairs * kExpertWidth));
    chk(dev_alloc(&L->h_lo, L->max_pairs * kExpertWidth));
    chk(dev_alloc(&L->ypart, (size_t)kDecodeChunks * kDecodeTile * d));
    chk(dev_alloc(&L->ecount, (size_t)E));
    chk(dev_alloc(&L->tokl, (size_t)E * max_tokens));
    L->pf_ncut = (max_tokens + kPfChunk - 1) / kPfChunk + 1;
    chk(dev_alloc(&L->pf_cut, (size_t)E * L->pf_ncut));
    chk(dev_alloc(&L->pf_ebase, (size_t)E));
    chk(dev_alloc(&L->plan, (size_t)4 + 4 * (size_t)plan_max_groups(L->dm, max_tokens) + E + 1));
    chk(dev_alloc(&L->dec_tok, (size_t)kDecodeTile * E));
    chk(dev_alloc(&L->emask, (size_t)E));
    if (a != hipSuccess) {
        free_layer(L);
        return hip_status(a);
    }
    chk(hipMemcpyAsync(L->Wr, W_r, dE * sizeof(uint16_t), hipMemcpyDeviceToDevice, s));
    if (router_bias)
        chk(hipMemcpyAsync(L->bias, router_bias, sizeof(float) * E, hipMemcpyDeviceToDevice, s));
    else
        chk(hipMemsetAsync(L->bias, 0, sizeof(float) * E, s));
    chk(hipMemsetAsync(L->counters, 0, sizeof(uint32_t) * L->n_counters, s));
    chk(hipMemsetAsync(L->emask, 0, sizeof(unsigned long long) * E, s));
    if (!gated && !b_fc) chk(hipMemsetAsync(L->bfc, 0, sizeof(float) * d_ff, s));
    if (L->bproj)
        chk(hipMemcpyAsync(L->bproj, b_proj, sizeof(float) * d, hipMemcpyDeviceToDevice, s));
    if (a == hipSuccess) a = launch_repack(L, W_gate, W_up, W_down, perm, gated ? nullptr : b_fc, s);
    chk(hipStreamSynchronize(s));
    if (a != hipSuccess) {
        free_layer(L);
        return hip_status(a);
    }
    *out = L;
    return PP_OK;
}

}  // namespace

extern "C" {

pp_status prunepath_create(pp_layer **out, int32_t d, int32_t d_ff, int32_t E,
                           int32_t max_tokens, const uint16_t *W_r, const uint16_t *W_gate,
                           const uint16_t *W_up, const uint16_t *W_down, const int32_t *perm,
                           const float *router_bias, uint32_t flags, void *hip_stream) {
    if (!out) return PP_EINVAL;
    *out = nullptr;
    if (!W_r || !W_gate || !W_up || !W_down) return PP_EINVAL;
    return create_layer(out, d, d_ff, E, max_tokens, W_r, W_gate, W_up, W_down, nullptr, nullptr,
                        perm, router_bias, flags, hip_stream);
}

pp_status prunepath_create_mlp(pp_layer **out, int32_t d, int32_t d_ff, int32_t E,
                               int32_t max_tokens, const uint16_t *W_r, const uint16_t *W_fc,
                               const float *b_fc, const uint16_t *W_proj, const float *b_proj,
                               const int32_t *perm, const float *router_bias, uint32_t flags,
                               void *hip_stream) {
    if (!out) return PP_EINVAL;
    *out = nullptr;
    if (!W_r || !W_fc || !W_proj) return PP_EINVAL;
    return create_layer(out, d, d_ff, E, max_tokens, W_r, W_fc, nullptr, W_proj, b_fc, b_proj,
                        perm, router_bias, flags, hip_stream);
}

pp_status prunepath_route(pp_layer *L, const uint16_t *x, int32_t T, float tau,
                          const float *inv_temp, int32_t *expert_idx, int32_t *count,
                          float *gate_w, void *hip_stream) {
    pp_status st = check_call(L, x, T, tau);
    if (st != PP_OK) return st;
    if (!expert_idx || !count) return PP_EINVAL;
    return hip_status(launch_route(L, x, T, tau, inv_temp, expert_idx, count, gate_w, false,
                                   static_cast<hipStream_t>(hip_stream)));
}

pp_status prunepath_ffn_decode(pp_layer *L, const uint16_t *x, int32_t T, float tau,
                               const float *inv_temp, float *y, int32_t *expert_idx,
                               int32_t *count, void *hip_stream) {
    return run_ffn(L, x, T, tau, inv_temp, y, expert_idx, count, hip_stream, false);
}

pp_status prunepath_ffn_prefill(pp_layer *L, const uint16_t *x, int32_t T, float tau,
                                const float *inv_temp, float *y, int32_t *expert_idx,
                                int32_t *count, void *hip_stream) {
    return run_ffn(L, x, T, tau, inv_temp, y, expert_idx, count, hip_stream, true);
}

pp_status prunepath_profile_begin(pp_layer *L, int32_t capacity) {
    if (!L || L->prof || capacity < 1 || capacity > (1 << 20)) return PP_EINVAL;
    profiler *P = new (std::nothrow) profiler;
    if (!P) return PP_ENOMEM;
    P->cap = capacity;
    P->ev.assign((size_t)2 * capacity, nullptr);
    P->kind.assign((size_t)capacity, 0);
    for (auto &e : P->ev) {
        if (hipEventCreate(&e) != hipSuccess) {
            e = nullptr;
            free_profiler(P);
            return PP_EHIP;
        }
    }
    L->prof = P;
    return PP_OK;
}

pp_status prunepath_profile_end(pp_layer *L, double *ms, int32_t *launches) {
    if (!L || !L->prof) return PP_EINVAL;
    profiler *P = L->prof;
    L->prof = nullptr;
    double acc[PP_KERNEL_COUNT] = {0, 0, 0, 0};
    int32_t n[PP_KERNEL_COUNT] = {0, 0, 0, 0};
    pp_status st = PP_OK;
    for (int i = 0; i < P->used && st == PP_OK; ++i) {
        float t = 0.f;
        if (hipEventSynchronize(P->ev[2 * i + 1]) != hipSuccess ||
            hipEventElapsedTime(&t, P->ev[2 * i], P->ev[2 * i + 1]) != hipSuccess) {
            st = PP_EHIP;
            break;
        }
        acc[P->kind[i]] += t;
        n[P->kind[i]] += 1;
    }
    free_profiler(P);
    for (int k = 0; k < PP_KERNEL_COUNT; ++k) {
        if (ms) ms[k] = acc[k];
        if (launches) launches[k] = n[k];
    }
    return st;
}

void prunepath_destroy(pp_layer *L) { free_layer(L); }

const char *prunepath_status_string(pp_status s) {
    switch (s) {
    case PP_OK: return "ok";
    case PP_EINVAL: return "invalid argument";
    case PP_ENOMEM: return "out of device memory";
    case PP_EHIP: return "HIP runtime error";
    case PP_EUNSUPPORTED: return "unsupported shape";
    case PP_ENOTCONVERGED: return "did not converge";
    }
    return "unknown status";
}

}  // extern "C"
