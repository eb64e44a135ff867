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
// HBM-bound: 12 B E bytes (g read twice, dg written once).  Three launches,
// each sum in an order fixed by (B, E), so results are deterministic:
//   loss_rows_k   64 rows per workgroup, staged in LDS by flat 16-byte loads;
//                 each row on the 16 lanes of one DPP row (4 rows per
//                 wavefront, no idle lanes when 16 divides E); per-workgroup
//                 column sums of p and entropy and sigmoid sums
//   loss_reduce_k one workgroup: workgroup partials in fp64 -> m and losses
//   loss_grad_k   16 rows per workgroup, staged the same way; dg is built in
//                 LDS and stored by flat 16-byte writes
// exp, log and reciprocal use the hardware instructions (1 ulp); kernels are
// instantiated for each ceil(E / 16).
#include <array>
#include <utility>

#include "pp_internal.h"

namespace pp {
namespace {

constexpr int kRowsWaves = 16;  // loss_rows_k: 64 rows per workgroup
constexpr int kGradWaves = 4;   // loss_grad_k: 16 rows per workgroup
constexpr int kLossRowsPerWave = 4;  // one row per 16-lane DPP row
constexpr int kRedThreads = 1024;
constexpr int kRedWaves = kRedThreads / 64;
constexpr int kRedBatch = 8;  // partial loads in flight per lane
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

// A workgroup of W wavefronts owns rows r0 .. r0 + 4W - 1 (r0 = 4W blockIdx.x),
// a contiguous range of 4W E floats.  It is copied into LDS with flat,
// coalesced 16-byte loads (all issued before the first LDS store), so the
// row length never decides the access pattern.  Wavefront w then takes the
// block's rows w, w + W, w + 2W, w + 3W.
template <int W>
struct Tile {
    static constexpr int kRows = kLossRowsPerWave * W;
    static constexpr int kThreads = 64 * W;
    static constexpr int kVec = kRows * kMaxExperts / 4 / kThreads;  // float4 per thread
    int r0, nr;

    // copy the block's rows of G into t; returns after a barrier
    __device__ void stage(const float *__restrict__ G, int B, int E, float *t) {
        r0 = blockIdx.x * kRows;
        nr = min(kRows, B - r0);
        const int n = nr * E, n4 = n >> 2;
        const float *src = G + (size_t)r0 * E;  // 16-byte aligned: r0 E is a multiple of 4
        const float4 *s4 = reinterpret_cast<const float4 *>(src);
        float4 *t4 = reinterpret_cast<float4 *>(t);
        if (n4 > 0) {  // workgroup-uniform
            // unconditional loads of clamped (in-range) addresses, so that all
            // of them are in flight before the first wait
            // (threads past the end copy the last vector again: same value,
            // same place), so no branch splits the loads from each other
            float4 v[kVec];
#pragma unroll
            for (int u = 0; u < kVec; ++u) v[u] = s4[min((int)threadIdx.x + kThreads * u, n4 - 1)];
#pragma unroll
            for (int u = 0; u < kVec; ++u) t4[min((int)threadIdx.x + kThreads * u, n4 - 1)] = v[u];
        }
        for (int i = 4 * n4 + threadIdx.x; i < n; i += kThreads) t[i] = src[i];
        __syncthreads();
    }
    // write the staged rows of t to D (after a barrier)
    __device__ void flush(const float *t, int E, float *__restrict__ D) const {
        __syncthreads();
        const int n = nr * E, n4 = n >> 2;
        float *dst = D + (size_t)r0 * E;
        if (n4 > 0) {
            const float4 *t4 = reinterpret_cast<const float4 *>(t);
            float4 *d4 = reinterpret_cast<float4 *>(dst);
            float4 v[kVec];
#pragma unroll
            for (int u = 0; u < kVec; ++u) v[u] = t4[min((int)threadIdx.x + kThreads * u, n4 - 1)];
#pragma unroll
            for (int u = 0; u < kVec; ++u) d4[min((int)threadIdx.x + kThreads * u, n4 - 1)] = v[u];
        }
        for (int i = 4 * n4 + threadIdx.x; i < n; i += kThreads) dst[i] = t[i];
    }
};

// One row of the tile on the 16 lanes of a DPP row: lane c holds columns
// c + 16 q, q < NQ = ceil(E / 16), and the row's softmax.  A row past the
// batch end (live false) reads row nr - 1 and must be ignored by the caller.
template <int NQ>
struct Row {
    float g[NQ], p[NQ];
    __device__ void load(const float *t, int lr, int nr, int E, int c) {
        const int rr = min(lr, nr - 1);
        float mx = -INFINITY;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = c + 16 * q;
            const float v = t[rr * E + min(j, E - 1)];
            g[q] = j < E ? v : -INFINITY;
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

// part: [nb][E + 2] = column sums of p over the block's 64 rows, then the
// block's sums of p log(p + eps) and of sigmoid(g); every sum runs over the
// rows in ascending order (in four quarters of 16 rows, then the quarters in
// order).
template <int NQ>
__global__ __launch_bounds__(64 * kRowsWaves) void loss_rows_k(const float *__restrict__ G, int B,
                                                               int E, float eps,
                                                               float *__restrict__ part) {
    using T = Tile<kRowsWaves>;
    __shared__ __align__(16) float tile[T::kRows * kMaxExperts];
    __shared__ float rows_es[2][T::kRows];
    __shared__ float quart[4][kMaxExperts + 2];
    const int lane = threadIdx.x & 63, c = lane & 15;
    const int lr = (threadIdx.x >> 6) * kLossRowsPerWave + (lane >> 4);
    T tl;
    tl.stage(G, B, E, tile);
    Row<NQ> R;
    R.load(tile, lr, tl.nr, E, c);
    float e = 0.0f, sg = 0.0f;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        if (c + 16 * q < E) {
            if (R.p[q] >= kFltMin) e += R.p[q] * flog(R.p[q] + eps);
            sg += fsig(R.g[q]);
        }
    }
    e = row16_sum(e);
    sg = row16_sum(sg);
    // a row's 16 lanes overwrite only their own row, which they have read
    const bool live = lr < tl.nr;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
        if (live && c + 16 * q < E) tile[lr * E + c + 16 * q] = R.p[q];
    if (c == 0) {
        rows_es[0][lr] = live ? e : 0.0f;
        rows_es[1][lr] = live ? sg : 0.0f;
    }
    __syncthreads();
    const int C = E + 2;
    for (int i = threadIdx.x; i < 4 * C; i += T::kThreads) {
        const int k = i / C, j = i - k * C;  // quarter k of the rows, column j
        const int r_end = min(tl.nr, 16 * k + 16);
        float v = 0.0f;
        for (int r = 16 * k; r < r_end; ++r)
            v += j < E ? tile[r * E + j] : rows_es[j - E][r];
        quart[k][j] = v;
    }
    __syncthreads();
    float *out = part + (size_t)blockIdx.x * C;
    for (int j = threadIdx.x; j < C; j += T::kThreads)
        out[j] = ((quart[0][j] + quart[1][j]) + quart[2][j]) + quart[3][j];
}

// One workgroup.  mout [E] = batch-mean probabilities; losses = [L_ent,
// L_bal, L_gate, L].  Wavefront w sums blocks w, w + 16, ... of each column
// in fp64; the 16 wavefront sums are then added in wavefront order, and
// sum_j m_j^2 is taken by wavefront 0 in a fixed butterfly.
__global__ __launch_bounds__(kRedThreads) void loss_reduce_k(const float *__restrict__ part, int nb,
                                                             int B, int E, float eta,
                                                             float lambda, float gamma,
                                                             float *__restrict__ mout,
                                                             float *__restrict__ losses) {
    __shared__ double red[kRedWaves][kMaxExperts + 2];
    __shared__ double col[kMaxExperts + 2];
    __shared__ double sq[kMaxExperts];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int C = E + 2;
    for (int c0 = 0; c0 < C; c0 += 64) {
        const int j = c0 + lane;
        if (j < C) {
            double acc = 0.0;
            for (int b0 = wv; b0 < nb; b0 += kRedWaves * kRedBatch) {
                float v[kRedBatch];
#pragma unroll
                for (int u = 0; u < kRedBatch; ++u) {
                    const int b = b0 + kRedWaves * u;
                    const float x = part[(size_t)min(b, nb - 1) * C + j];
                    v[u] = b < nb ? x : 0.0f;
                }
#pragma unroll
                for (int u = 0; u < kRedBatch; ++u) acc += (double)v[u];
            }
            red[wv][j] = acc;
        }
    }
    __syncthreads();
    const double invB = 1.0 / (double)B;
    for (int j = threadIdx.x; j < C; j += kRedThreads) {
        double v = red[0][j];
#pragma unroll
        for (int w = 1; w < kRedWaves; ++w) v += red[w][j];
        col[j] = v;
        if (j < E) {
            const double m = v * invB;
            mout[j] = (float)m;
            sq[j] = m * m;
        }
    }
    __syncthreads();
    if (wv == 0) {
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

// dg for the block's 16 rows (4 wavefronts x 4 rows): computed into the LDS
// tile in place of g, then stored with flat 16-byte writes.
template <int NQ>
__global__ __launch_bounds__(64 * kGradWaves) void loss_grad_k(const float *__restrict__ G, int B,
                                                               int E, float eps, float eta,
                                                               float lambda, float gamma,
                                                               const float *__restrict__ m,
                                                               float *__restrict__ dg) {
    using T = Tile<kGradWaves>;
    __shared__ __align__(16) float tile[T::kRows * kMaxExperts];
    const int lane = threadIdx.x & 63, c = lane & 15;
    const int lr = (threadIdx.x >> 6) * kLossRowsPerWave + (lane >> 4);
    const float ce = -eta / (float)B, cg = gamma / ((float)B * (float)E);
    const float cb = 2.0f * lambda * (float)E / (float)B;
    float bal[NQ];  // 2 lambda E m_j / B
#pragma unroll
    for (int q = 0; q < NQ; ++q) bal[q] = m[min(c + 16 * q, E - 1)];
#pragma unroll
    for (int q = 0; q < NQ; ++q) bal[q] = c + 16 * q < E ? cb * bal[q] : 0.0f;
    T tl;
    tl.stage(G, B, E, tile);
    Row<NQ> R;
    R.load(tile, lr, tl.nr, E, c);
    float a[NQ], pa = 0.0f;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const float pv = R.p[q];
        float ent = 0.0f;
        if (pv >= kFltMin) {
            const float pe = pv + eps;
            ent = ce * (flog(pe) + pv * frcp(pe));
        }
        a[q] = ent + bal[q];
        pa += pv * a[q];
    }
    pa = row16_sum(pa);
    if (lr < tl.nr) {  // a row's 16 lanes overwrite only their own row
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = c + 16 * q;
            if (j < E) {
                const float sv = fsig(R.g[q]);
                tile[lr * E + j] = R.p[q] * (a[q] - pa) + cg * sv * (1.0f - sv);
            }
        }
    }
    tl.flush(tile, E, dg);
}

inline int rows_blocks(int B) { return (B + Tile<kRowsWaves>::kRows - 1) / Tile<kRowsWaves>::kRows; }
inline int grad_blocks(int B) { return (B + Tile<kGradWaves>::kRows - 1) / Tile<kGradWaves>::kRows; }

template <int NQ>
void launch_loss(const float *g, int B, int E, float eps, float eta, float lambda, float gamma,
                 float *losses, float *dg, float *part, float *m, hipStream_t s) {
    const int nb = rows_blocks(B);
    hipLaunchKernelGGL(loss_rows_k<NQ>, dim3(nb), dim3(64 * kRowsWaves), 0, s, g, B, E, eps, part);
    hipLaunchKernelGGL(loss_reduce_k, dim3(1), dim3(kRedThreads), 0, s, part, nb, B, E, eta,
                       lambda, gamma, m, losses);
    if (dg)
        hipLaunchKernelGGL(loss_grad_k<NQ>, dim3(grad_blocks(B)), dim3(64 * kGradWaves), 0, s, g, B,
                           E, eps, eta, lambda, gamma, m, dg);
}

using LossLauncher = void (*)(const float *, int, int, float, float, float, float, float *,
                              float *, float *, float *, hipStream_t);
template <int... Q>
constexpr auto make_launchers(std::integer_sequence<int, Q...>) {
    return std::array<LossLauncher, sizeof...(Q)>{launch_loss<Q + 1>...};
}
constexpr auto kLaunchers = make_launchers(std::make_integer_sequence<int, kMaxExperts / 16>{});

}  // namespace
}  // namespace pp

extern "C" size_t prunepath_router_loss_workspace(int32_t B, int32_t E) {
    if (B < 1 || B > pp::kMaxLossRows || E < 1 || E > pp::kMaxExperts) return 0;
    return sizeof(float) * ((size_t)pp::rows_blocks(B) * ((size_t)E + 2) + (size_t)E);
}

extern "C" pp_status prunepath_router_loss(const float *g, int32_t B, int32_t E, float eps,
                                           float eta, float lambda, float gamma, float *losses,
                                           float *dg, void *workspace, void *hip_stream) {
    if (!g || !losses || !workspace || dg == g) return PP_EINVAL;
    if (B < 1 || B > pp::kMaxLossRows || E < 1 || E > pp::kMaxExperts) return PP_EINVAL;
    if (!(eps >= 0.0f && eps <= 3.0e38f) || !(fabsf(eta) <= 3.0e38f) ||
        !(fabsf(lambda) <= 3.0e38f) || !(fabsf(gamma) <= 3.0e38f))
        return PP_EINVAL;
    if (((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(dg)) & 15) ||
        ((reinterpret_cast<uintptr_t>(losses) | reinterpret_cast<uintptr_t>(workspace)) & 3))
        return PP_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    const int nb = pp::rows_blocks(B);
    float *part = static_cast<float *>(workspace);
    float *m = part + (size_t)nb * ((size_t)E + 2);
    pp::kLaunchers[(E + 15) / 16 - 1](g, B, E, eps, eta, lambda, gamma, losses, dg, part, m, s);
    return hipGetLastError() == hipSuccess ? PP_OK : PP_EHIP;
}
