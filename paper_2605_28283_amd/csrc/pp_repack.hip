// Create-time expert-major repack (Sec. 2.2: the permuted weights W Pi and
// Pi^T W_down, split into E contiguous experts of 128 neurons).
//
// The repacked layout stores every weight directly in the operand order of
// the gfx950 bf16 MFMA 16x16x32 (A operand: lane l holds row l%16, k-range
// 8*(l/16) .. +7 of a 16x32 tile), so each wavefront load in the FFN kernels
// is one contiguous, fully coalesced 1 KiB block:
//
//   Wgu: [e][nt = 0..7 neuron tiles of 16][s = 0..d/32-1][part: gate, up][lane][8]
//        element = W_part[n][32 s + 8 (lane/16) + j],  n = Pi(128 e + 16 nt + lane%16)
//        (a non-gated layer has the one part W_fc)
//   Wd:  [e][rt = 0..d/16-1 row tiles][s = 0..3][lane][8]
//        element = W_down[16 rt + lane%16][Pi(128 e + 32 s + 8 (lane/16) + j)]
//
// One expert's gate/up block is 2*128*d bf16 and its down block 128*d bf16,
// each contiguous.
#include "pp_internal.h"

namespace pp {
namespace {

__global__ void repack_gateup_k(const uint16_t *__restrict__ Wg, const uint16_t *__restrict__ Wu,
                                const int32_t *__restrict__ perm, int d, int NS, size_t nchunks,
                                uint16_t *__restrict__ out) {
    const int parts = Wu ? 2 : 1;
    for (size_t c = blockIdx.x * (size_t)blockDim.x + threadIdx.x; c < nchunks;
         c += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(c & 63);
        size_t r = c >> 6;
        const int part = parts == 2 ? (int)(r & 1) : 0;
        if (parts == 2) r >>= 1;
        const int s = (int)(r % NS);
        r /= NS;
        const int nt = (int)(r & 7);
        const size_t e = r >> 3;
        const size_t n0 = e * kExpertWidth + nt * 16 + (lane & 15);
        const size_t n = perm ? (size_t)perm[n0] : n0;
        const uint16_t *src = (part ? Wu : Wg) + n * d + s * kKStep + 8 * (lane >> 4);
        *reinterpret_cast<uint4 *>(out + c * 8) = *reinterpret_cast<const uint4 *>(src);
    }
}

__global__ void repack_down_k(const uint16_t *__restrict__ Wd, const int32_t *__restrict__ perm,
                              int d, int d_ff, size_t nchunks, uint16_t *__restrict__ out) {
    const int RT = d / 16;
    for (size_t c = blockIdx.x * (size_t)blockDim.x + threadIdx.x; c < nchunks;
         c += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(c & 63);
        size_t r = c >> 6;
        const int s = (int)(r & 3);
        r >>= 2;
        const int rt = (int)(r % RT);
        const size_t e = r / RT;
        const size_t row = (size_t)rt * 16 + (lane & 15);
        const size_t n0 = e * kExpertWidth + s * kKStep + 8 * (lane >> 4);
        uint16_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const size_t n = perm ? (size_t)perm[n0 + j] : n0 + j;
            v[j] = Wd[row * d_ff + n];
        }
        uint4 w;
        w.x = v[0] | ((uint32_t)v[1] << 16);
        w.y = v[2] | ((uint32_t)v[3] << 16);
        w.z = v[4] | ((uint32_t)v[5] << 16);
        w.w = v[6] | ((uint32_t)v[7] << 16);
        *reinterpret_cast<uint4 *>(out + c * 8) = w;
    }
}

// Input bias of a non-gated layer in expert order: out[i] = b[Pi(i)].
__global__ void repack_bias_k(const float *__restrict__ b, const int32_t *__restrict__ perm, int n,
                              float *__restrict__ out) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        out[i] = b[perm ? perm[i] : i];
}

}  // namespace

hipError_t launch_repack(pp_layer *L, const uint16_t *W_gate, const uint16_t *W_up,
                         const uint16_t *W_down, const int32_t *perm, const float *b_fc,
                         hipStream_t s) {
    const pp_dims &dm = L->dm;
    const size_t gu_chunks = (size_t)dm.E * 8 * dm.NS * (W_up ? 2 : 1) * 64;
    const size_t dn_chunks = (size_t)dm.E * (dm.d / 16) * 4 * 64;
    const int blk = 256;
    const int grid = 4 * L->num_cu * 8;
    hipLaunchKernelGGL(repack_gateup_k, dim3(grid), dim3(blk), 0, s, W_gate, W_up, perm, dm.d,
                       dm.NS, gu_chunks, L->Wgu);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(repack_down_k, dim3(grid), dim3(blk), 0, s, W_down, perm, dm.d, dm.d_ff,
                       dn_chunks, L->Wd);
    if (b_fc)
        hipLaunchKernelGGL(repack_bias_k, dim3((dm.d_ff + 255) / 256), dim3(256), 0, s, b_fc, perm,
                           dm.d_ff, L->bfc);
    return hipGetLastError();
}

}  // namespace pp
