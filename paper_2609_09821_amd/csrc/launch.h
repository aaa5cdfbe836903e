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
// Batches up to this many envs run the fused step on two threads per env when
// the skeleton has no path split (with the walks' prefetch ring, one thread
// per env is faster above it: 24576 and 32768 envs measured).
constexpr int64_t SPLIT_ENV_MAX = 16384;
// Batches up to this many envs run it on one thread per root-to-leaf path.
constexpr int64_t PATH_ENV_MAX = 16384;

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
    int x16_staged;      // non-zero: x16 already holds this observation (staged by an
                         // earlier layer of the same call), the staging pass is skipped
};

// The whole bf16 policy in one launch (policy_kernels.hip): hidden widths
// M_pad[l] multiples of 256 up to FUSED_MAX_WIDTH, observation width K_pad[0]
// up to FUSED_MAX_WIDTH, at most 128 padded actions.
constexpr int FUSED_MAX_LAYERS = 8;
constexpr int FUSED_MAX_WIDTH = 1024;

// Index of weight (o, i) of a bf16 [M_pad][K_pad] layer (K_pad = 64 nks) in
// MFMA fragment order: 1 KB blocks, one per (32-row tile t, K step ks of 64,
// substep s of 16), block b = (t nks + ks) 4 + s holding, for lane
// l = 32 h + r, the eight weights k = 64 ks + 16 s + 8 h .. +7 of row 32 t + r.
// A wavefront then loads the A operand of one MFMA as 1 KB of consecutive
// bytes, 16 per lane.
__host__ __device__ inline int64_t frag_index(int o, int i, int nks)
{
    const int t = o >> 5, r = o & 31, ks = i >> 6, s = (i >> 4) & 3, h = (i >> 3) & 1;
    return ((((int64_t)t * nks + ks) * 4 + s) * 64 + 32 * h + r) * 8 + (i & 7);
}

struct FusedMlpArgs {
    const float *obs;    // [D][ld_obs] fp32, env fastest
    int64_t ld_obs;
    uint32_t obs_bytes;  // D * ld_obs * 4
    int D;
    int L;
    const uint16_t *w[FUSED_MAX_LAYERS];   // M_pad x K_pad bf16 in fragment order (frag_index)
    const float *bias[FUSED_MAX_LAYERS];   // [M_pad]
    uint32_t w_bytes[FUSED_MAX_LAYERS];
    int M_pad[FUSED_MAX_LAYERS], K_pad[FUSED_MAX_LAYERS];
    GemmArgs out;        // sampling epilogue: N, bias (last layer), mean, action, logp,
                         // env_n, log_std, A, seed (a critic: N only)
    // a critic (launch_value_fused): the L layers are all hidden, then the value
    // v = head[0..M_pad[L-1]) . h + head[M_pad[L-1]] (fp32, zero past the width)
    const float *head;
    float *value;        // [N]
};
hipError_t launch_policy_fused(const FusedMlpArgs &f, hipStream_t s);
hipError_t launch_value_fused(const FusedMlpArgs &f, hipStream_t s);

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
                                  const float *bias, int64_t N, float *value, hipStream_t s);
hipError_t launch_value_head_obs(const float *obs, int64_t ld, int D, const float *w,
                                 const float *bias, bool bf16, int64_t N, float *value, hipStream_t s);
hipError_t launch_gae(const GaeArgs &g, hipStream_t s);
// Device address of im_gae_noalloc's scratch on `device`, which must be the
// current device (looked up on the first call per device, then cached).
hipError_t gae_scratch_address(int device, double **out);

// PPO update (train_kernels.hip).
enum { T_HIDDEN = 0, T_MASK = 1, T_LINEAR = 2, T_PARTIAL = 3 };

// C[m][n] = sum_k A[m][k] B(k, n) over whole 128 x 128 tiles; M, N multiples
// of 128, K and k_split of 64.
struct TGemm {
    const uint16_t *A;   // [M][lda] bf16, k contiguous
    int64_t lda;
    uint32_t a_bytes;
    const uint16_t *B;   // k-major [K][ldb] (n contiguous) or n-major [N][ldb]
    int64_t ldb;
    uint32_t b_bytes;
    int M, N, K, k_split;
    void *C;             // bf16 [M][ldc] (HIDDEN, MASK), fp32 [M][ldc] (LINEAR),
    int64_t ldc;         // fp32 [splits][M][ldc] (PARTIAL)
    const float *bias;   // [M] (HIDDEN, LINEAR)
    const uint16_t *mask;  // [M][ldm] bf16: the gradient passes where mask > 0 (MASK)
    int64_t ldm;
    int M_valid;         // LINEAR: rows written
    double *rs_part;     // MASK, optional: per-tile row sums of the stored (masked, bf16)
                         // output, rs_part[row * (N / tgemm_bn(N)) + column tile]
    uint4 *mbits;        // optional, 256x256 tiles only: the sign of the stored output as
                         // bits, tile-major.  HIDDEN writes them (bit = output > 0); MASK
                         // reads them instead of `mask` (the bits its M x N producer wrote)
};

// Column tile width of the training GEMM for N columns.
inline int tgemm_bn(int64_t N) { return N % 256 == 0 ? 256 : 128; }

struct GatherArgs {
    const float *obs;        // [T+1][D][ld]
    const float *action, *mean;  // [T][N][A]
    const float *logp, *adv_src, *ret_src, *value;  // [T][ld] ([T+1][ld] value)
    const int32_t *perm;     // chunk ids of this minibatch
    int chunks, chunks_pad;  // chunks of the minibatch, chunks covering Mb_pad
    int n_chunks;            // chunks of the rollout (perm entries are clamped to it)
    int64_t cpt, N, ld, Mb_pad;
    int D, K0, A;
    uint16_t *x0;            // [K0][Mb_pad] bf16
    float *act, *mean_old;   // [A][Mb_pad]
    float *logp_old, *adv, *ret, *vold;  // [Mb_pad]
};

constexpr int LOSS_STATS = 4;   // surrogate loss, value loss, KL, clip fraction
constexpr int MAX_ACTIONS = 128;  // widest policy output (action vector)

struct LossArgs {
    int64_t Mb, Mb_pad;
    int A;
    int64_t n_samples;              // advantages of the whole rollout (normalisation)
    const double *summary;          // IM_SUM_ADVANTAGE, IM_SUM_ADVANTAGE_SQ
    const float *mean, *act, *mean_old;   // [A][Mb_pad]
    const float *log_std, *log_std_old;   // [A]
    const float *logp_old, *adv, *ret, *vold, *value;  // [Mb_pad]
    float clip, value_coef;
    int clipped_value_loss;
    uint16_t *dmu;                  // [A][Mb_pad] bf16 out
    float *dv;                      // [Mb_pad] out
    double *partial;                // [blocks][A + LOSS_STATS]
};

struct LossReduceArgs {
    const double *partial;
    int blocks, A;
    int64_t Mb;
    float entropy_coef;
    float *grad_log_std;   // [A]
    double *mb_stats;      // [LOSS_STATS] minibatch means
};

struct OptScalars {
    float scale, lr, bc1, bc2;
};

struct FinalizeArgs {
    const double *norm_partial;
    int norm_blocks;
    const double *mb_stats;
    float max_grad_norm, desired_kl, lr_min, lr_max, beta1, beta2, eps;
    float *lr;             // device learning rate (adapted in place)
    int *step;             // device Adam step count
    OptScalars *opt;
    double *stats;         // IM_PPO_* sums or null
};

struct RepackArgs {
    const float *W, *b;    // masters [out][in], [out]
    int out, in;
    uint16_t *wt;          // [out..Mp][Kp] training copy or null
    uint16_t *wtt;         // [Kp][Mp] transposed training copy or null
    int Mp, Kp;
    void *roll;            // rollout copy [.][roll_K] or null
    int roll_K, roll_bf16; // 1: bf16, 2: fp32 of the bf16-rounded value, 0: fp32
    uint16_t *rollf;       // bf16 rollout copy in fragment order (frag_index, K_pad =
                           // roll_K) or null
    float *bias_train, *bias_roll;
};

hipError_t launch_tgemm(bool bt, int epi, const TGemm &g, int splits, hipStream_t s);
hipError_t launch_gather(const GatherArgs &a, hipStream_t s);
hipError_t launch_head_forward(const uint16_t *h, int K, int64_t Mb, const float *w, const float *b,
                               float *v, hipStream_t s);
// pw, pb (optional): [K][Mb / 2048] float64 partials of the head's weight
// gradient and of the rows' sums of the stored dz.
hipError_t launch_head_backward(const uint16_t *h, int K, int rows, int64_t Mb, const float *w,
                                const float *dv, uint16_t *dz, double *pw, double *pb, hipStream_t s);
// part: [rows][up to 2048 / rows + 1] float64 scratch
hipError_t launch_rowsum(bool bf16, const void *x, int rows, int64_t Mb, const float *y, double *part,
                         float *out, hipStream_t s);
// out[r] = sum over k < parts of part[r * parts + k] (float64, k in order), r < rows.
hipError_t launch_rowsum_finish(const double *part, int rows, int parts, float *out, hipStream_t s);
hipError_t launch_splitk_reduce(const float *P, int S, int64_t M, int64_t N, int rows, int cols,
                                float *out, hipStream_t s);
hipError_t launch_loss(const LossArgs &a, hipStream_t s);
hipError_t launch_loss_reduce(const LossReduceArgs &r, hipStream_t s);
hipError_t launch_optimizer(const float *grad, int64_t P, double *norm_partial, int norm_blocks,
                            const FinalizeArgs &f, float *x, float *m, float *v, hipStream_t s);
hipError_t launch_norm(const float *grad, int64_t P, double *norm_partial, int norm_blocks,
                       hipStream_t s);
hipError_t launch_repack(const RepackArgs &r, hipStream_t s);

hipError_t launch_env_step(int n_slots, int walk_slots, const EnvArgs &a, hipStream_t s);
hipError_t launch_reset(int n_slots, const EnvArgs &a, hipStream_t s);
hipError_t launch_standin(int n_slots, const EnvArgs &a, hipStream_t s);
hipError_t launch_pack_segments(const SkelTab *sk, int F, double fps, const float *root_pos,
                                const float *root_quat, const float *local_quat, float4 *seg,
                                hipStream_t s);
// *staged (if not null) is set when the layer read the observation through
// the bf16 staging buffer g.x16 (so that a later first layer on the same
// observation may pass x16_staged).
hipError_t launch_policy_layer(bool bf16, bool in_obs, bool sample, const GemmArgs &g, int M_pad,
                               hipStream_t s, bool *staged = nullptr);

}  // namespace im
