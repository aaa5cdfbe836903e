// launch.h -- argument blocks and host launchers shared by the C ABI layer
// and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tables.h"

namespace im {

// Batches up to this many envs use smaller GEMM tiles so that every layer
// still spreads over all 256 CUs.
constexpr int64_t SMALL_BATCH = 16384;
// Batches up to this many envs run the fused step on two threads per env.
constexpr int64_t SPLIT_ENV_MAX = 32768;

struct GemmArgs {
    const void *x;       // layer input: obs [K][ld_x] fp32 (first layer) or [N][ld_x] of T
    int64_t ld_x;
    const void *w;       // [M_pad][K_pad] of T
    const float *bias;   // [M_pad]
    int K_pad, K_valid;  // K_valid: rows of the observation that exist
    int64_t N;
    void *y;             // hidden output [N][ld_y] of T
    int64_t ld_y;
    // sampling epilogue
    float *mean, *action, *logp;
    const uint32_t *env_n;
    const float *log_std;
    int A;
    uint64_t seed;
    int M_blocks;        // feature blocks of the grid (set by the launcher)
    uint32_t w_bytes;    // extent of w in bytes (buffer-load bound)
    uint32_t x_bytes;    // extent of x in bytes: N * ld_x * elem, or D * ld_x * 4 for the observation
    void *x16;           // first bf16 layer of a large batch: [N][K_pad] bf16 staging of the
                         // observation (null: the GEMM reads the observation itself)
    int n_cu;            // compute units of the device (persistent grids)
    uint32_t y_bytes;    // extent of y in bytes (set by the launcher)
};

// Rollout end (rollout_kernels.hip).
struct GaeArgs {
    int T;
    int64_t n, ld;
    double gamma, lambda;
    const float *reward;
    const uint8_t *term, *trunc;
    const float *value;
    float *adv, *ret;
    float *ep_return;
    int32_t *ep_length;
    double *summary;      // null: no summaries
    double *partial;      // [blocks][IM_SUMMARY_FIELDS] per-block sums
};

hipError_t launch_value_head_rows(bool bf16, const void *x, int64_t ld_x, int K, const float *w,
                                  float bias, int64_t N, float *value, hipStream_t s);
hipError_t launch_value_head_obs(const float *obs, int64_t ld, int D, const float *w, float bias,
                                 bool bf16, int64_t N, float *value, hipStream_t s);
hipError_t launch_gae(const GaeArgs &g, hipStream_t s);

hipError_t launch_env_step(int n_slots, int half_slots, const EnvArgs &a, hipStream_t s);
hipError_t launch_reset(int n_slots, const EnvArgs &a, hipStream_t s);
hipError_t launch_standin(int n_slots, const EnvArgs &a, hipStream_t s);
hipError_t launch_pack_segments(const SkelTab *sk, int F, double fps, const float *root_pos,
                                const float *root_quat, const float *local_quat, float4 *seg,
                                hipStream_t s);
hipError_t launch_policy_layer(bool bf16, bool in_obs, bool sample, const GemmArgs &g, int M_pad,
                               hipStream_t s);

}  // namespace im
