// calib_kernels.hip -- measurement probes of the MI355X itself, not of the method.
//
// The rooflines the bench reports are priced against published peaks; these
// probes measure what the chip sustains for the same instruction mixes, so that
// a kernel's fraction of the peak can be read against what is reachable:
//   * MFMA: back-to-back v_mfma_f32_32x32x16_bf16 (the policy GEMMs' instruction)
//     or v_mfma_f32_32x32x2_f32, register operands only, 8 independent
//     accumulators per wave;
//   * LDS: ds_read_b128 / ds_read_b64 throughput per CU for 1..16 waves, in the
//     GEMM's fragment pattern (32 rows x 2 halves, XOR-swizzled 128-byte rows);
//   * global memory: a streaming 16-byte read of a buffer, once over a large
//     buffer (HBM) or many times over a small one (L2 / last-level cache).
// Every probe writes a checksum per wave so that nothing it computes is dead.
#include <hip/hip_runtime.h>

#include "instantmimic_calib.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int CHAINS = 8;

__global__ __launch_bounds__(256) void calib_mfma_bf16_kernel(int64_t iters, float *out)
{
    const int lane = threadIdx.x & 63;
    bf16x8_t a, b;
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(0.001f * (float)((lane + e) & 7));
        b[e] = (__bf16)(0.002f * (float)((lane * 3 + e) & 7));
    }
    f32x16_t acc[CHAINS];
    for (int c = 0; c < CHAINS; ++c)
        for (int r = 0; r < 16; ++r) acc[c][r] = 0.0f;
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
    }
    float s = 0.0f;
    for (int c = 0; c < CHAINS; ++c)
        for (int r = 0; r < 16; ++r) s += acc[c][r];
    out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void calib_mfma_f32_kernel(int64_t iters, float *out)
{
    const int lane = threadIdx.x & 63;
    const float a = 0.001f * (float)(lane & 7), b = 0.002f * (float)((lane * 3) & 7);
    f32x16_t acc[CHAINS];
    for (int c = 0; c < CHAINS; ++c)
        for (int r = 0; r < 16; ++r) acc[c][r] = 0.0f;
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
    }
    float s = 0.0f;
    for (int c = 0; c < CHAINS; ++c)
        for (int r = 0; r < 16; ++r) s += acc[c][r];
    out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// One block per CU; each wave issues 16 reads per round trip and waits for
// them.  Offsets stay inside the 64 KB array (row < 512, 128-byte rows).
template <int WIDTH>
__global__ __launch_bounds__(1024) void calib_lds_kernel(int64_t iters, uint32_t *out)
{
    __shared__ __attribute__((aligned(1024))) uint8_t lds[65536];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int i = tid; i < 65536 / 4; i += blockDim.x) ((uint32_t *)lds)[i] = (uint32_t)i * 2654435761u;
    __syncthreads();
    uint32_t x = 0;
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            int off;
            if (WIDTH == 16) {
                // the GEMM's fragment read: row r, 16-byte chunk q ^ ((r / 2) % 8)
                const int r = (wave * 32 + s * 8 + (lane & 31)) & 511;
                const int q = (2 * (s & 3) + (lane >> 5)) & 7;
                off = r * 128 + ((q ^ ((r >> 1) & 7)) * 16);
            } else {
                // 8 bytes per lane, consecutive lanes consecutive
                off = ((wave * 16 + s) * 512 + lane * 8) & 65535;
            }
            // opaque offset: the reads cannot be hoisted out of the loop
            asm volatile("" : "+v"(off));
            if (WIDTH == 16) {
                const u32x4_t v = *(const u32x4_t *)(lds + off);
                x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
            } else {
                const u32x2_t v = *(const u32x2_t *)(lds + off);
                x ^= v[0] ^ v[1];
            }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    }
    out[(int64_t)blockIdx.x * blockDim.x + tid] = x;
}

// Streaming read: thread t of the grid reads 16-byte words t, t + T, ... of
// `words` words, `passes` times over.
__global__ __launch_bounds__(256) void calib_read_kernel(const u32x4_t *__restrict__ src, int64_t words,
                                                         int passes, uint32_t *out)
{
    const int64_t T = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t x = 0;
    for (int p = 0; p < passes; ++p)
        for (int64_t w = t0; w < words; w += T) {
            const u32x4_t v = src[w];
            x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
        }
    out[t0] = x;
}

inline im_status launched() { return hipGetLastError() == hipSuccess ? IM_OK : IM_ERR_HIP; }

}  // namespace

extern "C" {

im_status im_calib_mfma(int kind, int64_t iters, int blocks, float *out, void *stream)
{
    if ((kind != IM_CALIB_MFMA_BF16 && kind != IM_CALIB_MFMA_F32) || iters < 1 || blocks < 1 || !out)
        return IM_ERR_INVALID_ARG;
    hipStream_t s = (hipStream_t)stream;
    if (kind == IM_CALIB_MFMA_BF16)
        hipLaunchKernelGGL(calib_mfma_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, s, iters, out);
    else
        hipLaunchKernelGGL(calib_mfma_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, iters, out);
    return launched();
}

im_status im_calib_lds(int width, int waves, int64_t iters, int blocks, uint32_t *out, void *stream)
{
    if ((width != 8 && width != 16) || waves < 1 || waves > 16 || iters < 1 || blocks < 1 || !out)
        return IM_ERR_INVALID_ARG;
    hipStream_t s = (hipStream_t)stream;
    if (width == 16)
        hipLaunchKernelGGL(calib_lds_kernel<16>, dim3((unsigned)blocks), dim3(64 * waves), 0, s, iters, out);
    else
        hipLaunchKernelGGL(calib_lds_kernel<8>, dim3((unsigned)blocks), dim3(64 * waves), 0, s, iters, out);
    return launched();
}

im_status im_calib_read(const void *src, int64_t bytes, int passes, int blocks, uint32_t *out, void *stream)
{
    if (!src || !out || bytes < 16 || (bytes & 15) || ((uintptr_t)src & 15) || passes < 1 || blocks < 1)
        return IM_ERR_INVALID_ARG;
    hipLaunchKernelGGL(calib_read_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                       (const u32x4_t *)src, bytes / 16, passes, out);
    return launched();
}

}  // extern "C"
