// rollout_kernels.hip -- the rollout end of the PPO loop (Fig. 3): the value
// head of the critic, generalized advantage estimation over the rollout
// storage and the rollout summaries, all on the device (Sec. 4: training
// summaries stay on the GPU, nothing is read back during the rollout).
//
// Storage layout: every per-step array is [T][ld] (env fastest), so a
// wavefront of 64 consecutive envs moves 256 contiguous bytes per step.
#include <hip/hip_runtime.h>

#include <mutex>

#include "device_math.h"
#include "launch.h"

namespace im {

// ---------------------------------------------------------------------------
// Scratch of im_gae_noalloc: the per-block summary sums ([blocks][fields]
// float64, one block per 256 envs) in a fixed device array instead of the
// context's buffer, so that the call allocates nothing.  Every device the
// library runs on holds one copy (320 KiB) until the process ends; all calls
// on a device share it.
// ---------------------------------------------------------------------------
constexpr int64_t GAE_SCRATCH_DOUBLES = (IM_GAE_NOALLOC_MAX_ENVS / 256) * IM_SUMMARY_FIELDS;
static __device__ __align__(256) double gae_scratch[GAE_SCRATCH_DOUBLES];

hipError_t gae_scratch_address(int device, double **out)
{
    // In host code `gae_scratch` only stands for the symbol: its device
    // address (different on every device) comes from the runtime, once per
    // device, with that device current.
    constexpr int MAX_DEVICES = 64;
    static std::mutex mu;
    static double *addr[MAX_DEVICES] = {};
    if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(gae_scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[device] = (double *)p;
    }
    *out = addr[device];
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// Value head, last layer: value[e] = b[0] + sum_k w[k] x[e][k] over the last
// hidden activations x [N][ld_x] (bf16 or fp32 rows, zero beyond the layer's
// width).  16 lanes per env, each reading 16-byte pieces of the row (256
// contiguous bytes per env and step of the loop); the 16 partial sums meet
// in a fixed butterfly, so the result does not depend on timing.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ __launch_bounds__(256) void value_head_rows_kernel(const void *__restrict__ x,
                                                              int64_t ld_x, int K,
                                                              const float *__restrict__ w,
                                                              const float *__restrict__ bias,
                                                              int64_t N, float *__restrict__ value)
{
    constexpr int EPC = BF16 ? 8 : 4;   // elements per 16-byte piece
    const int sub = threadIdx.x & 15;
    const int64_t e = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    float acc = 0.0f;
    if (e < N) {
        const int n_chunks = K / EPC;
        const char *row = (const char *)x + (size_t)e * (size_t)ld_x * (BF16 ? 2 : 4);
        for (int c = sub; c < n_chunks; c += 16) {
            const uint4 v = *(const uint4 *)(row + (size_t)c * 16);
            const float4 *wc = (const float4 *)(w + (size_t)c * EPC);
            if constexpr (BF16) {
                const float4 w0 = wc[0], w1 = wc[1];
                acc += w0.x * bf16_to_f32((uint16_t)(v.x & 0xFFFF));
                acc += w0.y * bf16_to_f32((uint16_t)(v.x >> 16));
                acc += w0.z * bf16_to_f32((uint16_t)(v.y & 0xFFFF));
                acc += w0.w * bf16_to_f32((uint16_t)(v.y >> 16));
                acc += w1.x * bf16_to_f32((uint16_t)(v.z & 0xFFFF));
                acc += w1.y * bf16_to_f32((uint16_t)(v.z >> 16));
                acc += w1.z * bf16_to_f32((uint16_t)(v.w & 0xFFFF));
                acc += w1.w * bf16_to_f32((uint16_t)(v.w >> 16));
            } else {
                const float4 w0 = wc[0];
                acc += w0.x * __uint_as_float(v.x);
                acc += w0.y * __uint_as_float(v.y);
                acc += w0.z * __uint_as_float(v.z);
                acc += w0.w * __uint_as_float(v.w);
            }
        }
    }
    acc += __shfl_xor(acc, 8, 16);
    acc += __shfl_xor(acc, 4, 16);
    acc += __shfl_xor(acc, 2, 16);
    acc += __shfl_xor(acc, 1, 16);
    if (e < N && sub == 0) value[e] = acc + bias[0];
}

// Value head of a one-layer critic: value[e] = b + sum_i w[i] obs[i][e] over
// the observation [D][ld] (rounded to bf16 first for a bf16 critic).
__global__ __launch_bounds__(256) void value_head_obs_kernel(const float *__restrict__ obs,
                                                             int64_t ld, int D,
                                                             const float *__restrict__ w,
                                                             const float *__restrict__ bias, int bf16,
                                                             int64_t N, float *__restrict__ value)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= N) return;
    float acc = 0.0f;
    for (int i = 0; i < D; ++i) {
        float v = obs[(int64_t)i * ld + e];
        if (bf16) v = bf16_to_f32(f32_to_bf16_rne(v));
        acc += w[i] * v;
    }
    value[e] = acc + bias[0];
}

// ---------------------------------------------------------------------------
// GAE and summaries.  One thread per env walks its column of the storage:
// forward for the episode bookkeeping, backward for the advantage recursion
//   delta_t = r_t + gamma * next_t - V_t,  next_t = 0 (terminated),
//             V_t (truncated only), V_{t+1} (otherwise)
//   A_t = delta_t + gamma * lambda * A_{t+1} (0 past an episode end or the
//         rollout end),  R_t = A_t + V_t,
// in float64 (no contraction: the same operations in the same order as the
// recursion written out), stored as float32.  The per-thread sums of the
// summary fields are reduced per block in a fixed tree, and across blocks by
// summary_reduce_kernel in block order.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gae_kernel(GaeArgs g)
{
    // steps are read in chunks of C, two chunk buffers in turn: the loads of
    // the next chunk are issued before the current one is processed (and,
    // backwards, before its stores -- a wave counts loads and stores in one
    // in-order queue, so loads issued after stores wait for them).  The loop
    // is unrolled by two so that each buffer keeps its registers.  Steps
    // outside [0, T) load step 0 or T - 1 and are not processed.
    constexpr int C = 8;
    __shared__ double red[IM_SUMMARY_FIELDS][256];
    const int tid = threadIdx.x;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + tid;
    double s[IM_SUMMARY_FIELDS];
#pragma unroll
    for (int f = 0; f < IM_SUMMARY_FIELDS; ++f) s[f] = 0.0;
    if (e < g.n) {
        const int64_t ld = g.ld;
        const int T = g.T;
        if (g.summary) {
            float epr = g.ep_return[e];
            int32_t epl = g.ep_length[e];
            float ra[C], rb[C];
            uint8_t ta[C], tb[C], ua[C], ub[C];
            auto load_fwd = [&](int t0, float (&r)[C], uint8_t (&te)[C], uint8_t (&tr)[C]) {
#pragma unroll
                for (int j = 0; j < C; ++j) {
                    const int t = t0 + j < T ? t0 + j : T - 1;
                    const int64_t i = (int64_t)t * ld + e;
                    r[j] = g.reward[i];
                    te[j] = g.term[i];
                    tr[j] = g.trunc[i];
                }
            };
            auto fwd = [&](int t0, const float (&r)[C], const uint8_t (&te)[C], const uint8_t (&tr)[C]) {
#pragma unroll
                for (int j = 0; j < C; ++j) {
                    if (t0 + j >= T) break;
                    s[IM_SUM_REWARD] += (double)r[j];
                    {
#pragma clang fp contract(off)
                        epr = epr + r[j];
                    }
                    epl += 1;
                    s[IM_SUM_TERMINATED] += te[j] ? 1.0 : 0.0;
                    s[IM_SUM_TRUNCATED] += tr[j] ? 1.0 : 0.0;
                    if (te[j] || tr[j]) {
                        s[IM_SUM_EPISODES] += 1.0;
                        s[IM_SUM_EPISODE_RETURN] += (double)epr;
                        s[IM_SUM_EPISODE_LENGTH] += (double)epl;
                        epr = 0.0f;
                        epl = 0;
                    }
                }
            };
            load_fwd(0, ra, ta, ua);
            for (int t0 = 0; t0 < T; t0 += 2 * C) {
                load_fwd(t0 + C, rb, tb, ub);
                fwd(t0, ra, ta, ua);
                load_fwd(t0 + 2 * C, ra, ta, ua);
                if (t0 + C < T) fwd(t0 + C, rb, tb, ub);
            }
            g.ep_return[e] = epr;
            g.ep_length[e] = epl;
        }
        {
#pragma clang fp contract(off)
            const double gam = g.gamma, gl = g.gamma * g.lambda;
            double adv = 0.0;
            double v_next = (double)g.value[(int64_t)T * ld + e];
            float ra[C], rb[C], va[C], vb[C];
            uint8_t ta[C], tb[C], ua[C], ub[C];
            // chunk ending at step t1 - 1, walked backwards (j = 0 is step t1 - 1)
            auto load_bwd = [&](int t1, float (&r)[C], float (&v)[C], uint8_t (&te)[C],
                                uint8_t (&tr)[C]) {
#pragma unroll
                for (int j = 0; j < C; ++j) {
                    const int t = t1 - 1 - j >= 0 ? t1 - 1 - j : 0;
                    const int64_t i = (int64_t)t * ld + e;
                    r[j] = g.reward[i];
                    v[j] = g.value[i];
                    te[j] = g.term[i];
                    tr[j] = g.trunc[i];
                }
            };
            auto bwd = [&](int t1, const float (&r)[C], const float (&v)[C], const uint8_t (&te)[C],
                           const uint8_t (&tr)[C]) {
#pragma unroll
                for (int j = 0; j < C; ++j) {
                    const int t = t1 - 1 - j;
                    if (t < 0) break;
                    const int64_t i = (int64_t)t * ld + e;
                    const double vt = (double)v[j];
                    const double nxt = te[j] ? 0.0 : (tr[j] ? vt : v_next);
                    const double delta = ((double)r[j] + gam * nxt) - vt;
                    adv = (te[j] || tr[j]) ? delta : delta + gl * adv;
                    const float a32 = (float)adv;
                    const float r32 = (float)(adv + vt);
                    g.adv[i] = a32;
                    g.ret[i] = r32;
                    s[IM_SUM_ADVANTAGE] += (double)a32;
                    s[IM_SUM_ADVANTAGE_SQ] += (double)a32 * (double)a32;
                    s[IM_SUM_VALUE] += vt;
                    s[IM_SUM_RETURN] += (double)r32;
                    v_next = vt;
                }
            };
            load_bwd(T, ra, va, ta, ua);
            for (int t1 = T; t1 > 0; t1 -= 2 * C) {
                load_bwd(t1 - C, rb, vb, tb, ub);
                bwd(t1, ra, va, ta, ua);
                load_bwd(t1 - 2 * C, ra, va, ta, ua);
                if (t1 - C > 0) bwd(t1 - C, rb, vb, tb, ub);
            }
        }
    }
    if (!g.summary) return;   // uniform over the grid
#pragma unroll
    for (int f = 0; f < IM_SUMMARY_FIELDS; ++f) red[f][tid] = s[f];
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (tid < h) {
#pragma unroll
            for (int f = 0; f < IM_SUMMARY_FIELDS; ++f) red[f][tid] += red[f][tid + h];
        }
        __syncthreads();
    }
    if (tid < IM_SUMMARY_FIELDS) g.partial[(int64_t)blockIdx.x * IM_SUMMARY_FIELDS + tid] = red[tid][0];
}

// One block: thread j sums the partials of blocks j, j + 256, ... in order,
// then a fixed tree over the threads.
__global__ __launch_bounds__(256) void summary_reduce_kernel(const double *__restrict__ partial,
                                                             int n_blocks, double *__restrict__ out)
{
    __shared__ double red[IM_SUMMARY_FIELDS][256];
    const int tid = threadIdx.x;
    double s[IM_SUMMARY_FIELDS];
#pragma unroll
    for (int f = 0; f < IM_SUMMARY_FIELDS; ++f) s[f] = 0.0;
    for (int b = tid; b < n_blocks; b += 256)
#pragma unroll
        for (int f = 0; f < IM_SUMMARY_FIELDS; ++f) s[f] += partial[(int64_t)b * IM_SUMMARY_FIELDS + f];
#pragma unroll
    for (int f = 0; f < IM_SUMMARY_FIELDS; ++f) red[f][tid] = s[f];
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (tid < h) {
#pragma unroll
            for (int f = 0; f < IM_SUMMARY_FIELDS; ++f) red[f][tid] += red[f][tid + h];
        }
        __syncthreads();
    }
    if (tid < IM_SUMMARY_FIELDS) out[tid] = red[tid][0];
}

// ---------------------------------------------------------------------------
// Host-side launchers.
// ---------------------------------------------------------------------------
hipError_t launch_value_head_rows(bool bf16, const void *x, int64_t ld_x, int K, const float *w,
                                  const float *bias, int64_t N, float *value, hipStream_t s)
{
    if (N <= 0) return hipSuccess;
    const dim3 grid((unsigned)((N + 15) / 16));
    if (bf16)
        hipLaunchKernelGGL(value_head_rows_kernel<true>, grid, dim3(256), 0, s, x, ld_x, K, w, bias,
                           N, value);
    else
        hipLaunchKernelGGL(value_head_rows_kernel<false>, grid, dim3(256), 0, s, x, ld_x, K, w, bias,
                           N, value);
    return hipGetLastError();
}

hipError_t launch_value_head_obs(const float *obs, int64_t ld, int D, const float *w,
                                 const float *bias, bool bf16, int64_t N, float *value, hipStream_t s)
{
    if (N <= 0) return hipSuccess;
    hipLaunchKernelGGL(value_head_obs_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, s,
                       obs, ld, D, w, bias, bf16 ? 1 : 0, N, value);
    return hipGetLastError();
}

hipError_t launch_gae(const GaeArgs &g, hipStream_t s)
{
    const int64_t blocks = (g.n + 255) / 256;
    if (g.n > 0)
        hipLaunchKernelGGL(gae_kernel, dim3((unsigned)blocks), dim3(256), 0, s, g);
    if (g.summary)   // zero envs: the reduction of no blocks writes zeros
        hipLaunchKernelGGL(summary_reduce_kernel, dim3(1), dim3(256), 0, s, g.partial, (int)blocks,
                           g.summary);
    return hipGetLastError();
}

}  // namespace im
