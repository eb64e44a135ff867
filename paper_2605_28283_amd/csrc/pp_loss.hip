// Routing regularisers of PrunePath's training objective, forward and
// backward, over a batch of router logits g [B, E] (fp32, row-major):
//   p_ij   = softmax_j(g_i)                                 Eq. (softmax_prob)
//   L_ent  = -(1/B) sum_i sum_j p_ij log(p_ij + eps)        Eq. (entropy_loss), Sec. 3.2
//   L_bal  = E sum_j m_j^2,  m_j = (1/B) sum_i p_ij         Eq. (load_balance_loss), Sec. 3.2
//   L_gate = (1/(B E)) sum_ij sigmoid(g_ij)                 gate-magnitude term, Sec. 4.2.3
//   L      = eta L_ent + lambda L_bal + gamma L_gate        Eq. (train_loss) plus that term
// and dL/dg.  With a_ij = dL/dp_ij = -(eta/B) (log(p_ij + eps) + p_ij/(p_ij + eps))
// + 2 lambda E m_j / B, the softmax backward contracts to
//   dL/dg_ij = p_ij (a_ij - sum_k p_ik a_ik) + (gamma/(B E)) s_ij (1 - s_ij),
// s = sigmoid(g).  A term with p_ij = 0 (eps = 0 and an underflowed
// probability) is taken at its limit, 0.
//
// HBM-bound: 12 B E bytes (g read twice, dg written once).  Two launches,
// each sum in an order fixed by (B, E), so results are deterministic:
//   loss_rows_k   each row on the 16 lanes of one DPP row (4 rows per
//                 wavefront, no idle lanes when 16 divides E), 64 rows per
//                 workgroup; per-workgroup column sums of p and entropy and
//                 sigmoid sums
//   loss_grad_k   every workgroup reduces those partials in fp64 to m (the
//                 gradient of L_bal needs the batch mean), workgroup 0 writes
//                 the losses; then dg for 64 rows in the same row layout,
//                 written straight from registers
// exp, log and reciprocal use the hardware instructions (1 ulp); kernels are
// instantiated for each ceil(E / 16).
#include <array>
#include <atomic>
#include <mutex>
#include <utility>

#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kLossWaves = 16;       // wavefronts per workgroup, both kernels
constexpr int kLossRowsPerWave = 4;  // one row per 16-lane DPP row
constexpr int kRowsPerBlock = kLossWaves * kLossRowsPerWave;  // 64
constexpr int kRedLoads = 32;  // partial loads in flight per lane in the reduction
constexpr int kMaxLossRows = 1 << 22;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kFltMin = 1.17549435e-38f;  // smallest normal binary32

// Hardware transcendentals (1 ulp on their own argument): e^x as 2^(x log2 e),
// ln x as log2(x) ln 2, 1/x.  A term p log p with p below the smallest
// normal number is taken as 0 (|p log p| < 1e-36).
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float flog(float x) { return __builtin_amdgcn_logf(x) * kLn2; }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float fsig(float g) { return frcp(1.0f + fexp(-g)); }

// Butterflies over the 16 lanes of a DPP row (quad swaps, then the half-row
// and row mirrors); every lane ends with the same value, since each step adds
// the same two operands on both partners.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_sum(float v) {
    v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp<0x141>(v);  // row_half_mirror
    v += dpp<0x140>(v);  // row_mirror
    return v;
}
__device__ __forceinline__ float row16_max(float v) {
    v = fmaxf(v, dpp<0xB1>(v));
    v = fmaxf(v, dpp<0x4E>(v));
    v = fmaxf(v, dpp<0x141>(v));
    v = fmaxf(v, dpp<0x140>(v));
    return v;
}

// Row r on the 16 lanes of one DPP row: lane c holds columns c + 16 q,
// q < NQ = ceil(E / 16), and the row's softmax.  Rows are read straight from
// HBM, 4 consecutive rows per wavefront (one 16-lane segment of 64 bytes per
// row and instruction), every load unconditional (clamped address) so all of
// them are in flight before the first wait.  A row past the batch end reads
// row B - 1 and must be ignored by the caller.
template <int NQ>
struct Row {
    float g[NQ], p[NQ];
    // issue the row's loads (no wait)
    __device__ void fetch(const float *__restrict__ G, int r, int B, int E, int c) {
        const float *row = G + (size_t)min(r, B - 1) * E;
#pragma unroll
        for (int q = 0; q < NQ; ++q) g[q] = row[min(c + 16 * q, E - 1)];
    }
    __device__ void softmax(int E, int c) {
        float mx = -INFINITY;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            g[q] = c + 16 * q < E ? g[q] : -INFINITY;
            mx = fmaxf(mx, g[q]);
        }
        mx = row16_max(mx);
        float s = 0.0f;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            p[q] = fexp(g[q] - mx);  // 0 for the padding columns
            s += p[q];
        }
        const float inv = 1.0f / row16_sum(s);
#pragma unroll
        for (int q = 0; q < NQ; ++q) p[q] *= inv;
    }
};

// Sum over the four 16-lane rows of a wavefront, (r0 + r1) + (r2 + r3) in
// every lane.
__device__ __forceinline__ float wave_rows_sum(float v, int lane) {
    v += __uint_as_float(xor_lane<16>(__float_as_uint(v), lane));
    v += __uint_as_float(xor_lane<32>(__float_as_uint(v), lane));
    return v;
}

// part: [nb][E + 2] = column sums of p over each workgroup's 64 rows, then
// its sums of p log(p + eps) and of sigmoid(g).  Fixed order: within a
// wavefront (r0 + r1) + (r2 + r3), then the 16 wavefronts in order.
template <int NQ>
__global__ __launch_bounds__(64 * kLossWaves) void loss_rows_k(const float *__restrict__ G, int B,
                                                               int E, float eps,
                                                               float *__restrict__ part) {
    __shared__ float ws[kLossWaves][kMaxExperts + 2];
    const int lane = threadIdx.x & 63, c = lane & 15, wv = threadIdx.x >> 6;
    const int r = blockIdx.x * kRowsPerBlock + wv * kLossRowsPerWave + (lane >> 4);
    const bool live = r < B;
    Row<NQ> R;
    R.fetch(G, r, B, E, c);
    R.softmax(E, c);
    float e = 0.0f, sg = 0.0f;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const float pv = live ? R.p[q] : 0.0f;
        if (pv >= kFltMin) e += pv * flog(pv + eps);
        if (live && c + 16 * q < E) sg += fsig(R.g[q]);
        R.p[q] = wave_rows_sum(pv, lane);
    }
    e = wave_rows_sum(row16_sum(e), lane);
    sg = wave_rows_sum(row16_sum(sg), lane);
    if (lane < 16) {
#pragma unroll
        for (int q = 0; q < NQ; ++q)
            if (c + 16 * q < E) ws[wv][c + 16 * q] = R.p[q];
        if (c == 0) {
            ws[wv][E] = e;
            ws[wv][E + 1] = sg;
        }
    }
    __syncthreads();
    float *out = part + (size_t)blockIdx.x * (E + 2);
    for (int j = threadIdx.x; j < E + 2; j += 64 * kLossWaves) {
        float v = ws[0][j];
#pragma unroll
        for (int w = 1; w < kLossWaves; ++w) v += ws[w][j];
        out[j] = v;
    }
}

// The reduction of all nb partial rows, run by every workgroup of
// loss_grad_k (it needs m) -- 117 KB for the 16384 x 112 batch, read from L2
// after the first workgroup of an XCD has fetched it.  Wavefront w sums
// partial rows w, w + 16, ... of each column in fp64 (NC = ceil((E + 2) / 64)
// columns per lane, 32 / NC partial rows per round, all loads of a round in
// flight at once); the 16 wavefront sums are added in wavefront order.
// mf [E] receives m_j (fp32); workgroup 0 also writes losses = [L_ent,
// L_bal, L_gate, L] (sum_j m_j^2 by a fixed butterfly in wavefront 0).
// Every workgroup takes the same steps in the same order, so all hold the
// same m.
template <int NC>
__device__ void reduce_partials(const float *__restrict__ part, int nb, int B, int E, float eta,
                                float lambda, float gamma, float *mf,
                                float *__restrict__ losses) {
    __shared__ double red[kLossWaves][kMaxExperts + 2];
    __shared__ double col[kMaxExperts + 2];
    __shared__ double sq[kMaxExperts];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int C = E + 2;
    constexpr int RB = kRedLoads / NC;  // partial rows per round
    double acc[NC] = {};
    for (int b0 = wv; b0 < nb; b0 += kLossWaves * RB) {
        float v[RB][NC];
#pragma unroll
        for (int u = 0; u < RB; ++u)
#pragma unroll
            for (int k = 0; k < NC; ++k)
                v[u][k] = part[(size_t)min(b0 + kLossWaves * u, nb - 1) * C + min(lane + 64 * k, C - 1)];
#pragma unroll
        for (int u = 0; u < RB; ++u)
#pragma unroll
            for (int k = 0; k < NC; ++k)
                acc[k] += b0 + kLossWaves * u < nb ? (double)v[u][k] : 0.0;
    }
#pragma unroll
    for (int k = 0; k < NC; ++k)
        if (lane + 64 * k < C) red[wv][lane + 64 * k] = acc[k];
    __syncthreads();
    const double invB = 1.0 / (double)B;
    for (int j = threadIdx.x; j < C; j += 64 * kLossWaves) {
        double v = red[0][j];
#pragma unroll
        for (int w = 1; w < kLossWaves; ++w) v += red[w][j];
        col[j] = v;
        if (j < E) {
            const double m = v * invB;
            mf[j] = (float)m;
            sq[j] = m * m;
        }
    }
    __syncthreads();
    if (blockIdx.x == 0 && wv == 0) {
        double s = 0.0;
#pragma unroll
        for (int q = 0; q < kMaxExperts / 64; ++q)
            if (lane + 64 * q < E) s += sq[lane + 64 * q];
#pragma unroll
        for (int st = 32; st >= 1; st >>= 1) s += __shfl_xor(s, st, 64);
        if (lane == 0) {
            const double l_ent = -col[E] * invB;
            const double l_bal = (double)E * s;
            const double l_gate = col[E + 1] * invB / (double)E;
            losses[0] = (float)l_ent;
            losses[1] = (float)l_bal;
            losses[2] = (float)l_gate;
            losses[3] =
                (float)((double)eta * l_ent + (double)lambda * l_bal + (double)gamma * l_gate);
        }
    }
}

// dg, 64 rows per workgroup (4 per wavefront), straight from registers to
// HBM.  The rows' loads are issued before the partials are reduced, so their
// HBM latency overlaps the reduction.  With dg NULL the kernel runs as one
// workgroup that only writes the losses.
template <int NQ, int NC>
__global__ __launch_bounds__(64 * kLossWaves) void loss_grad_k(const float *__restrict__ G, int B,
                                                               int E, float eps, float eta,
                                                               float lambda, float gamma,
                                                               const float *__restrict__ part,
                                                               int nb, float *__restrict__ losses,
                                                               float *__restrict__ dg) {
    __shared__ float mf[kMaxExperts];
    const int lane = threadIdx.x & 63, c = lane & 15;
    const int r = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6) * kLossRowsPerWave + (lane >> 4);
    Row<NQ> R;
    if (dg) R.fetch(G, r, B, E, c);
    reduce_partials<NC>(part, nb, B, E, eta, lambda, gamma, mf, losses);
    if (!dg) return;
    const float ce = -eta / (float)B, cg = gamma / ((float)B * (float)E);
    const float cb = 2.0f * lambda * (float)E / (float)B;
    R.softmax(E, c);
    float a[NQ], pa = 0.0f;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const float pv = R.p[q];
        float ent = 0.0f;
        if (pv >= kFltMin) {
            const float pe = pv + eps;
            ent = ce * (flog(pe) + pv * frcp(pe));
        }
        a[q] = ent + (c + 16 * q < E ? cb * mf[min(c + 16 * q, E - 1)] : 0.0f);
        pa += pv * a[q];
    }
    pa = row16_sum(pa);
    if (r < B) {
        float *out = dg + (size_t)r * E;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = c + 16 * q;
            if (j < E) {
                const float sv = fsig(R.g[q]);
                out[j] = R.p[q] * (a[q] - pa) + cg * sv * (1.0f - sv);
            }
        }
    }
}

inline int rows_blocks(int B) { return (B + kRowsPerBlock - 1) / kRowsPerBlock; }

template <int NQ, int NC>
void launch_loss_nc(const float *g, int B, int E, float eps, float eta, float lambda, float gamma,
                    float *losses, float *dg, float *part, hipStream_t s) {
    const int nb = rows_blocks(B);
    hipLaunchKernelGGL(loss_rows_k<NQ>, dim3(nb), dim3(64 * kLossWaves), 0, s, g, B, E, eps, part);
    hipLaunchKernelGGL((loss_grad_k<NQ, NC>), dim3(dg ? nb : 1), dim3(64 * kLossWaves), 0, s, g, B,
                       E, eps, eta, lambda, gamma, part, nb, losses, dg);
}

// NC = ceil((E + 2) / 64) follows from NQ = ceil(E / 16) except at the
// boundaries E = 63, 127, 191, 255 (E + 2 crosses a multiple of 64).
template <int NQ>
void launch_loss(const float *g, int B, int E, float eps, float eta, float lambda, float gamma,
                 float *losses, float *dg, float *part, hipStream_t s) {
    constexpr int lo = (16 * (NQ - 1) + 1 + 2 + 63) / 64, hi = (16 * NQ + 2 + 63) / 64;
    if ((E + 2 + 63) / 64 == lo)
        launch_loss_nc<NQ, lo>(g, B, E, eps, eta, lambda, gamma, losses, dg, part, s);
    else
        launch_loss_nc<NQ, hi>(g, B, E, eps, eta, lambda, gamma, losses, dg, part, s);
}

using LossLauncher = void (*)(const float *, int, int, float, float, float, float, float *,
                              float *, float *, hipStream_t);
template <int... Q>
constexpr auto make_launchers(std::integer_sequence<int, Q...>) {
    return std::array<LossLauncher, sizeof...(Q)>{launch_loss<Q + 1>...};
}
constexpr auto kLaunchers = make_launchers(std::make_integer_sequence<int, kMaxExperts / 16>{});

}  // namespace
}  // namespace pp

// ---------------------------------------------- allocation-free variant
// The partials of prunepath_router_loss_noalloc live in this file-scope
// device array (one copy per GPU, held until the process ends).  In host code
// the name `scratch` is a host-side stand-in, not a device address: kernels
// take the address hipGetSymbolAddress returns on each device, kept in
// g_scratch_dev.
constexpr size_t kLossScratchBytes = PP_ROUTER_LOSS_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) float scratch[kLossScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<float *> g_scratch_dev[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of `scratch` on the current device, resolved on the first
// call on each device and kept.
pp_status loss_scratch_address(float **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return PP_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return PP_EUNSUPPORTED;
    float *p = g_scratch_dev[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_dev[dev].load(std::memory_order_relaxed);
        if (!p) {
            void *a = nullptr;
            if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || !a) return PP_EHIP;
            p = static_cast<float *>(a);
            g_scratch_dev[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return PP_OK;
}

// Argument checks shared by both entry points (workspace aside).
pp_status check_loss_args(const float *g, int32_t B, int32_t E, float eps, float eta,
                          float lambda, float gamma, const float *losses, const float *dg) {
    if (!g || !losses || dg == g) return PP_EINVAL;
    if (B < 1 || B > pp::kMaxLossRows || E < 1 || E > pp::kMaxExperts) return PP_EINVAL;
    if (!(eps >= 0.0f && eps <= 3.0e38f) || !(fabsf(eta) <= 3.0e38f) ||
        !(fabsf(lambda) <= 3.0e38f) || !(fabsf(gamma) <= 3.0e38f))
        return PP_EINVAL;
    if (((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(dg)) & 15) ||
        (reinterpret_cast<uintptr_t>(losses) & 3))
        return PP_EINVAL;
    return PP_OK;
}
}  // namespace

extern "C" size_t prunepath_router_loss_workspace(int32_t B, int32_t E) {
    if (B < 1 || B > pp::kMaxLossRows || E < 1 || E > pp::kMaxExperts) return 0;
    return sizeof(float) * (size_t)pp::rows_blocks(B) * ((size_t)E + 2);
}

extern "C" pp_status prunepath_router_loss(const float *g, int32_t B, int32_t E, float eps,
                                           float eta, float lambda, float gamma, float *losses,
                                           float *dg, void *workspace, void *hip_stream) {
    pp_status st = check_loss_args(g, B, E, eps, eta, lambda, gamma, losses, dg);
    if (st != PP_OK) return st;
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 3)) return PP_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    pp::kLaunchers[(E + 15) / 16 - 1](g, B, E, eps, eta, lambda, gamma, losses, dg,
                                      static_cast<float *>(workspace), s);
    return hipGetLastError() == hipSuccess ? PP_OK : PP_EHIP;
}

extern "C" pp_status prunepath_router_loss_noalloc(const float *g, int32_t B, int32_t E,
                                                   float eps, float eta, float lambda,
                                                   float gamma, float *losses, float *dg,
                                                   void *hip_stream) {
    pp_status st = check_loss_args(g, B, E, eps, eta, lambda, gamma, losses, dg);
    if (st != PP_OK) return st;
    if (prunepath_router_loss_workspace(B, E) > kLossScratchBytes) return PP_EUNSUPPORTED;
    float *ws = nullptr;
    st = loss_scratch_address(&ws);
    if (st != PP_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    // the kernels overwrite every partial they read: nothing to clear
    pp::kLaunchers[(E + 15) / 16 - 1](g, B, E, eps, eta, lambda, gamma, losses, dg, ws, s);
    return hipGetLastError() == hipSuccess ? PP_OK : PP_EHIP;
}
