// policy_kernels.hip -- Gaussian MLP policy on the CDNA4 matrix cores.
//
// Each layer is one GEMM  Y[N][M] = act(X[N][K] W[M][K]^T + b)  run on MFMA
// 32x32 tiles: A operand = weight rows (output features), B operand = envs.
// Accumulator lane l of a 32x32 tile holds column (env) l % 32 and, for
// register r, row 8 (r / 4) + 4 (l / 32) + r % 4, i.e. four consecutive
// output features per register group.  That gives each lane whole groups of
// four actions in the last layer, which is exactly one Philox block of
// action noise.
//
// bf16 path: v_mfma_f32_32x32x16_bf16, the observation is rounded to bf16
// while it is staged, hidden activations are stored as bf16.  fp32 path:
// v_mfma_f32_32x32x2_f32 with fp32 activations.  Accumulation is fp32.
//
// The first layer reads the observation in its [D][ld] (env-fastest)
// layout and transposes it into LDS; hidden activations are stored env-major
// ([N][M_pad], feature-fastest) so later layers stage both operands with
// contiguous K runs.
#include <hip/hip_runtime.h>

#include "device_math.h"
#include "launch.h"

namespace im {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float HALF_LOG_2PI = 0.91893853320467274f;

template <bool BF16>
struct Elem;
template <>
struct Elem<true> {
    using T = uint16_t;
    static constexpr int KSTEP = 16;  // K of one MFMA
};
template <>
struct Elem<false> {
    using T = float;
    static constexpr int KSTEP = 2;
};

// Tile: WGM x WGN waves, each MT x NT MFMA tiles of 32x32; K chunk KC.
template <bool BF16, bool IN_OBS, bool SAMPLE, int WGM, int WGN, int MT, int NT>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_layer_kernel(GemmArgs g)
{
    using T = typename Elem<BF16>::T;
    constexpr int KSTEP = Elem<BF16>::KSTEP;
    constexpr int KC = 32;
    constexpr int BM = WGM * MT * 32, BN = WGN * NT * 32;
    constexpr int NTHR = 64 * WGM * WGN;
    constexpr int PAD = 16 / sizeof(T);  // 16-byte row padding against bank conflicts
    constexpr int LDA = KC + PAD;

    __shared__ __attribute__((aligned(16))) T As[BM * LDA];
    __shared__ __attribute__((aligned(16))) T Bs[BN * LDA];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int64_t n0 = (int64_t)blockIdx.y * BN;
    const T *W = (const T *)g.w;

    f32x16_t acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    for (int k0 = 0; k0 < g.K_pad; k0 += KC) {
        // ---- stage the weight tile (rows contiguous in K) ----
        {
            constexpr int VEC = 16 / sizeof(T);          // elements per 16-byte load
            constexpr int PER_ROW = KC / VEC;
            for (int v = tid; v < BM * PER_ROW; v += NTHR) {
                const int r = v / PER_ROW, c = (v % PER_ROW) * VEC;
                const uint4 q = *(const uint4 *)(W + (m0 + r) * g.K_pad + k0 + c);
                *(uint4 *)(&As[r * LDA + c]) = q;
            }
        }
        // ---- stage the activation tile ----
        if constexpr (IN_OBS) {
            const float *X = (const float *)g.x;
            for (int v = tid; v < BN * KC; v += NTHR) {
                const int kk = v / BN, nn = v % BN;
                const int k = k0 + kk;
                const int64_t n = n0 + nn;
                float val = 0.0f;
                if (k < g.K_valid && n < g.N) val = X[(int64_t)k * g.ld_x + n];
                if constexpr (BF16)
                    Bs[nn * LDA + kk] = f32_to_bf16_rne(val);
                else
                    Bs[nn * LDA + kk] = val;
            }
        } else {
            const T *X = (const T *)g.x;
            constexpr int VEC = 16 / sizeof(T);
            constexpr int PER_ROW = KC / VEC;
            for (int v = tid; v < BN * PER_ROW; v += NTHR) {
                const int r = v / PER_ROW, c = (v % PER_ROW) * VEC;
                const int64_t n = n0 + r;
                uint4 q = make_uint4(0u, 0u, 0u, 0u);
                if (n < g.N) q = *(const uint4 *)(X + n * g.ld_x + k0 + c);
                *(uint4 *)(&Bs[r * LDA + c]) = q;
            }
        }
        __syncthreads();

        // ---- MFMA over the chunk ----
#pragma unroll
        for (int ks = 0; ks < KC; ks += KSTEP) {
            if constexpr (BF16) {
                bf16x8_t af[MT], bfr[NT];
                const int kof = ks + 8 * (lane >> 5);
#pragma unroll
                for (int i = 0; i < MT; ++i) {
                    const int row = (wm * MT + i) * 32 + (lane & 31);
                    af[i] = *(const bf16x8_t *)(&As[row * LDA + kof]);
                }
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                    const int row = (wn * NT + j) * 32 + (lane & 31);
                    bfr[j] = *(const bf16x8_t *)(&Bs[row * LDA + kof]);
                }
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j],
                                                                            acc[i][j], 0, 0, 0);
            } else {
                float af[MT], bfr[NT];
                const int kof = ks + (lane >> 5);
#pragma unroll
                for (int i = 0; i < MT; ++i) {
                    const int row = (wm * MT + i) * 32 + (lane & 31);
                    af[i] = As[row * LDA + kof];
                }
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                    const int row = (wn * NT + j) * 32 + (lane & 31);
                    bfr[j] = Bs[row * LDA + kof];
                }
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bfr[j], acc[i][j],
                                                                         0, 0, 0);
            }
        }
        __syncthreads();
    }

    // ---- epilogues ----
    if constexpr (!SAMPLE) {
        T *Y = (T *)g.y;
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const int64_t n = n0 + (wn * NT + j) * 32 + (lane & 31);
                if (n >= g.N) continue;
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) {
                    const int64_t m = m0 + (wm * MT + i) * 32 + 8 * grp + 4 * (lane >> 5);
                    float v[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float y = acc[i][j][4 * grp + q] + g.bias[m + q];
                        v[q] = y > 0.0f ? y : 0.0f;
                    }
                    if constexpr (BF16) {
                        const uint32_t lo = (uint32_t)f32_to_bf16_rne(v[0]) |
                                            ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
                        const uint32_t hi = (uint32_t)f32_to_bf16_rne(v[2]) |
                                            ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
                        *(uint2 *)(Y + n * g.ld_y + m) = make_uint2(lo, hi);
                    } else {
                        *(float4 *)(Y + n * g.ld_y + m) = make_float4(v[0], v[1], v[2], v[3]);
                    }
                }
            }
    } else {
        // the block covers every action (m0 == 0); NT == 1
        const int64_t n = n0 + wn * 32 + (lane & 31);
        const bool valid_n = n < g.N;
        float lp = 0.0f;
        const uint32_t en = valid_n ? g.env_n[n] : 0u;
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const int mb = i * 32 + 8 * grp + 4 * (lane >> 5);
                if (!valid_n || mb >= g.A) continue;
                float z[4];
                normals4(g.seed, (uint32_t)n, en, (uint32_t)(mb >> 2), 0u, z);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int m = mb + q;
                    if (m < g.A) {
                        const float mu = acc[i][0][4 * grp + q] + g.bias[m];
                        const float ls = g.log_std[m];
                        g.mean[n * g.A + m] = mu;
                        g.action[n * g.A + m] = mu + expf(ls) * z[q];
                        lp += 0.5f * z[q] * z[q] + ls + HALF_LOG_2PI;
                    }
                }
            }
        lp += __shfl_xor(lp, 32);
        if (valid_n && lane < 32 && g.logp) g.logp[n] = -lp;
    }
}

template <bool BF16, bool IN_OBS>
static hipError_t launch_hidden(const GemmArgs &g, int M_pad, hipStream_t s)
{
    constexpr int WGM = 2, WGN = 2, MT = 2, NT = 2;
    const dim3 grid((unsigned)(M_pad / (WGM * MT * 32)),
                    (unsigned)((g.N + WGN * NT * 32 - 1) / (WGN * NT * 32)));
    hipLaunchKernelGGL((gemm_layer_kernel<BF16, IN_OBS, false, WGM, WGN, MT, NT>), grid,
                       dim3(64 * WGM * WGN), 0, s, g);
    return hipGetLastError();
}

template <bool BF16, bool IN_OBS, int MT>
static hipError_t launch_sample_mt(const GemmArgs &g, hipStream_t s)
{
    constexpr int WGN = 4;
    const dim3 grid(1u, (unsigned)((g.N + WGN * 32 - 1) / (WGN * 32)));
    hipLaunchKernelGGL((gemm_layer_kernel<BF16, IN_OBS, true, 1, WGN, MT, 1>), grid,
                       dim3(64 * WGN), 0, s, g);
    return hipGetLastError();
}

template <bool BF16, bool IN_OBS>
static hipError_t launch_sample(const GemmArgs &g, int M_pad, hipStream_t s)
{
    switch (M_pad / 32) {
        case 1: return launch_sample_mt<BF16, IN_OBS, 1>(g, s);
        case 2: return launch_sample_mt<BF16, IN_OBS, 2>(g, s);
        case 3: return launch_sample_mt<BF16, IN_OBS, 3>(g, s);
        default: return launch_sample_mt<BF16, IN_OBS, 4>(g, s);
    }
}

// Host entry used by the C ABI layer: one layer.
hipError_t launch_policy_layer(bool bf16, bool in_obs, bool sample, const GemmArgs &g, int M_pad,
                               hipStream_t s)
{
    if (g.N <= 0) return hipSuccess;
    if (!sample) {
        if (bf16) return in_obs ? launch_hidden<true, true>(g, M_pad, s) : launch_hidden<true, false>(g, M_pad, s);
        return in_obs ? launch_hidden<false, true>(g, M_pad, s) : launch_hidden<false, false>(g, M_pad, s);
    }
    if (bf16) return in_obs ? launch_sample<true, true>(g, M_pad, s) : launch_sample<true, false>(g, M_pad, s);
    return in_obs ? launch_sample<false, true>(g, M_pad, s) : launch_sample<false, false>(g, M_pad, s);
}

}  // namespace im
