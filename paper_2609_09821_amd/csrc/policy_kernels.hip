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
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr float HALF_LOG_2PI = 0.91893853320467274f;


// Writes n_valid*A consecutive floats from LDS to dst (16-byte stores when dst
// is 16-byte aligned).
template <int NTHR>
__device__ __forceinline__ void copy_rows_out(float *dst, const float *so, int64_t cnt, int tid)
{
    if ((((uintptr_t)dst) & 15) == 0) {
        const int64_t c4 = cnt >> 2;
        for (int64_t v = tid; v < c4; v += NTHR)
            *(f32x4_t *)(dst + 4 * v) = *(const f32x4_t *)(so + 4 * v);
        for (int64_t v = 4 * c4 + tid; v < cnt; v += NTHR) dst[v] = so[v];
    } else {
        for (int64_t v = tid; v < cnt; v += NTHR) dst[v] = so[v];
    }
}

// Epilogue of the last layer: mean = acc + b, Gaussian noise from Philox, action
// = mean + exp(log_std) z, logp (sigma and the noise-free part of logp are
// formed once per block).  The accumulators follow the 32x32 MFMA layout
// (lane column = env, rows 8*grp + 4*(lane/32) + q = actions); the block covers
// every action of its envs (m0 == 0).  The block's envs n0 .. n0+nv-1 own the
// contiguous ranges mean[n0*A .. (n0+nv)*A) and action[...], so both are staged
// in LDS (`so`, at least BN*A floats, free once the main loop has ended with a
// barrier) and written out with wide stores; the accumulators are reused to hold
// the actions between the two passes.
template <int NTHR, int TM, int TN>
__device__ __forceinline__ void sample_epilogue(const GemmArgs &g, float *so, int64_t n0, int64_t nv,
                                                int col0, int tid, f32x16_t (&acc)[TM][TN])
{
    const int lane = tid & 63;
    const int A = g.A;
    // Once per block, in LDS: the biases and sigma = exp(log_std) of every
    // action (each lane's values then add an LDS read, not a global load in
    // its own divergent branch), and the noise-free part of -logp, the sum over
    // actions of log_std + log(2 pi) / 2, by wave 0 in a fixed butterfly.
    __shared__ float sig[TM * 32];
    __shared__ float sbias[TM * 32];
    __shared__ float lp0;
    for (int m = tid; m < A; m += NTHR) {
        sig[m] = expf(g.log_std[m]);
        sbias[m] = g.bias[m];
    }
    if (tid < 64) {
        float c = 0.0f;
        for (int m = tid; m < A; m += 64) c += g.log_std[m] + HALF_LOG_2PI;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
        if (tid == 0) lp0 = c;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int nl = col0 + j * 32 + (lane & 31);
        const int64_t n = n0 + nl;
        const bool valid_n = nl < nv;
        const uint32_t en = valid_n ? g.env_n[n] : 0u;
        float lp = 0.0f;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const int mb = i * 32 + 8 * grp + 4 * (lane >> 5);
                if (!valid_n || mb >= A) continue;
                float z[4];
                normals4(g.seed, (uint32_t)n, en, (uint32_t)(mb >> 2), 0u, z);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int m = mb + q;
                    if (m < A) {
                        const float mu = acc[i][j][4 * grp + q] + sbias[m];
                        so[nl * A + m] = mu;
                        acc[i][j][4 * grp + q] = mu + sig[m] * z[q];
                        lp += 0.5f * z[q] * z[q];
                    }
                }
            }
        lp += __shfl_xor(lp, 32);
        if (valid_n && lane < 32 && g.logp) g.logp[n] = -(lp + lp0);
    }
    __syncthreads();
    copy_rows_out<NTHR>(g.mean + n0 * A, so, nv * A, tid);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int nl = col0 + j * 32 + (lane & 31);
        if (nl >= nv) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const int mb = i * 32 + 8 * grp + 4 * (lane >> 5);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (mb + q < A) so[nl * A + mb + q] = acc[i][j][4 * grp + q];
            }
    }
    __syncthreads();
    copy_rows_out<NTHR>(g.action + n0 * A, so, nv * A, tid);
}

// fp32 layer GEMM.  Tile: WGM x WGN waves, each MT x NT MFMA tiles of 32x32
// (v_mfma_f32_32x32x2_f32); K chunk 32.  16-byte global loads into
// registers one chunk ahead, two LDS buffers, one barrier per chunk.  The
// first layer reads the observation [D][ld] (env fastest) with 16-byte loads
// along envs and transposes it into LDS.
template <bool IN_OBS, bool SAMPLE, int WGM, int WGN, int MT, int NT>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_f32_kernel(GemmArgs g)
{
    constexpr int KC = 32;
    constexpr int BM = WGM * MT * 32, BN = WGN * NT * 32;
    constexpr int NTHR = 64 * WGM * WGN;
    constexpr int LDA = KC + 4;                  // floats per LDS row (16-byte pad)
    constexpr int STAGE = (BM + BN) * LDA;
    constexpr int A_CH = BM * (KC / 4) / NTHR;   // float4 chunks of the weight tile per thread
    constexpr int B_CH = BN * (KC / 4) / NTHR;   // hidden input: float4 chunks per thread
    constexpr int O_CH = KC * (BN / 4) / NTHR;   // observation: float4 (4 envs of one k) per thread
    static_assert(BM * (KC / 4) % NTHR == 0 && BN * (KC / 4) % NTHR == 0 && KC * (BN / 4) % NTHR == 0, "split");

    // the sampling epilogue reuses the stage buffers for a BN x A output tile
    constexpr int LDS_FLOATS = (SAMPLE && BN * BM > 2 * STAGE) ? BN * BM : 2 * STAGE;
    __shared__ __attribute__((aligned(16))) float lds[LDS_FLOATS];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int64_t n0 = (int64_t)blockIdx.y * BN;
    const float *W = (const float *)g.w;
    const float *X = (const float *)g.x;
    // raw buffer loads: past the extent they return zero (env tail, rows of
    // the observation beyond D); columns past N inside the extent only feed
    // accumulator columns that are never stored
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)X, (short)0, (int)g.x_bytes, 0x00020000);
    const bool vec_obs = IN_OBS && ((g.ld_x & 3) == 0) && ((((uintptr_t)X) & 15) == 0);
    (void)vec_obs;

    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)W, (short)0, (int)g.w_bytes, 0x00020000);
    // three register stages: the global loads of chunk k+3 go out while chunk
    // k is multiplied and chunk k+1 (loaded two chunks earlier) is stored to LDS
    constexpr int RB = IN_OBS ? O_CH : B_CH;
    f32x4_t ra0[A_CH], rb0[RB], ra1[A_CH], rb1[RB], ra2[A_CH], rb2[RB];
    auto load_global = [&](int k0, f32x4_t (&ra)[A_CH], f32x4_t (&rb)[RB]) {
#pragma unroll
        for (int c = 0; c < A_CH; ++c) {
            const int v = tid + c * NTHR;
            const int r = v / (KC / 4), q = v % (KC / 4);
            const uint32_t off = (uint32_t)(((m0 + r) * g.K_pad + k0 + q * 4) * 4);
            ra[c] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, off, 0, 0));
        }
        if constexpr (!IN_OBS) {
#pragma unroll
            for (int c = 0; c < B_CH; ++c) {
                const int v = tid + c * NTHR;
                const int r = v / (KC / 4), q = v % (KC / 4);
                const uint32_t off = (uint32_t)(((n0 + r) * g.ld_x + k0 + q * 4) * 4);
                rb[c] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
            }
        } else {
#pragma unroll
            for (int c = 0; c < O_CH; ++c) {
                const int v = tid + c * NTHR;
                const int kk = v / (BN / 4), nq = (v % (BN / 4)) * 4;
                const uint32_t off = (uint32_t)((((int64_t)(k0 + kk)) * g.ld_x + n0 + nq) * 4);
                if (vec_obs) {
                    rb[c] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
                } else {
                    rb[c][0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0));
                    rb[c][1] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xr, off + 4, 0, 0));
                    rb[c][2] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xr, off + 8, 0, 0));
                    rb[c][3] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xr, off + 12, 0, 0));
                }
            }
        }
    };
    auto store_lds = [&](int buf, const f32x4_t (&ra)[A_CH], const f32x4_t (&rb)[RB]) {
        float *As = lds + buf * STAGE;
        float *Bs = As + BM * LDA;
#pragma unroll
        for (int c = 0; c < A_CH; ++c) {
            const int v = tid + c * NTHR;
            *(f32x4_t *)(As + (v / (KC / 4)) * LDA + (v % (KC / 4)) * 4) = ra[c];
        }
        if constexpr (!IN_OBS) {
#pragma unroll
            for (int c = 0; c < B_CH; ++c) {
                const int v = tid + c * NTHR;
                *(f32x4_t *)(Bs + (v / (KC / 4)) * LDA + (v % (KC / 4)) * 4) = rb[c];
            }
        } else {
#pragma unroll
            for (int c = 0; c < O_CH; ++c) {
                const int v = tid + c * NTHR;
                const int kk = v / (BN / 4), nq = (v % (BN / 4)) * 4;
                Bs[(nq + 0) * LDA + kk] = rb[c][0];
                Bs[(nq + 1) * LDA + kk] = rb[c][1];
                Bs[(nq + 2) * LDA + kk] = rb[c][2];
                Bs[(nq + 3) * LDA + kk] = rb[c][3];
            }
        }
    };

    f32x16_t acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // MFMA 4t + q of a chunk takes, in each half h = lane / 32 of the wave,
    // element q of the 16-byte run at k = 8t + 4h (operands A and B alike), so
    // one 16-byte LDS read per operand feeds four MFMAs.  Rows of 36 floats put
    // 16 consecutive rows of one run on distinct bank groups.
    auto compute = [&](int buf) {
        const float *As = lds + buf * STAGE;
        const float *Bs = As + BM * LDA;
        const int arow = wm * (MT * 32) + (lane & 31), brow = wn * (NT * 32) + (lane & 31);
        const int kh = 4 * (lane >> 5);
#pragma unroll
        for (int t = 0; t < KC / 8; ++t) {
            f32x4_t af[MT], bfr[NT];
#pragma unroll
            for (int i = 0; i < MT; ++i) af[i] = *(const f32x4_t *)(As + (arow + i * 32) * LDA + 8 * t + kh);
#pragma unroll
            for (int j = 0; j < NT; ++j) bfr[j] = *(const f32x4_t *)(Bs + (brow + j * 32) * LDA + 8 * t + kh);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i][q], bfr[j][q], acc[i][j], 0, 0, 0);
        }
    };

    const int nk = g.K_pad / KC;
    load_global(0, ra0, rb0);
    store_lds(0, ra0, rb0);
    __syncthreads();
    if (nk > 1) load_global(KC, ra1, rb1);
    if (nk > 2) load_global(2 * KC, ra2, rb2);
    // chunk kt: registers of chunk kt+1 in stage (kt+1) % 3, loads of kt+3 into
    // stage kt % 3 (stored to LDS in the previous iteration)
    auto step = [&](int kt, const f32x4_t (&sa)[A_CH], const f32x4_t (&sb)[RB], f32x4_t (&la)[A_CH],
                    f32x4_t (&lb)[RB]) {
        compute(kt & 1);
        if (kt + 1 < nk) store_lds((kt + 1) & 1, sa, sb);
        if (kt + 3 < nk) load_global((kt + 3) * KC, la, lb);
        __syncthreads();
    };
    for (int kt = 0; kt < nk; kt += 3) {
        step(kt, ra1, rb1, ra0, rb0);
        if (kt + 1 < nk) step(kt + 1, ra2, rb2, ra1, rb1);
        if (kt + 2 < nk) step(kt + 2, ra0, rb0, ra2, rb2);
    }

    if constexpr (!SAMPLE) {
        float *Y = (float *)g.y;
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const int64_t n = n0 + (wn * NT + j) * 32 + (lane & 31);
                if (n >= g.N) continue;
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) {
                    const int64_t m = m0 + (wm * MT + i) * 32 + 8 * grp + 4 * (lane >> 5);
                    const float4 bb = *(const float4 *)(g.bias + m);
                    *(float4 *)(Y + n * g.ld_y + m) =
                        make_float4(fmaxf(acc[i][j][4 * grp + 0] + bb.x, 0.0f),
                                    fmaxf(acc[i][j][4 * grp + 1] + bb.y, 0.0f),
                                    fmaxf(acc[i][j][4 * grp + 2] + bb.z, 0.0f),
                                    fmaxf(acc[i][j][4 * grp + 3] + bb.w, 0.0f));
                }
            }
    } else {
        // the block covers every action (m0 == 0)
        const int64_t nv = g.N - n0 < BN ? g.N - n0 : BN;
        sample_epilogue<NTHR, MT, NT>(g, lds, n0, nv, wn * NT * 32, tid, acc);
    }
}

// Last fp32 layer + sampling for small batches: one column of 32 envs and all
// MT x 32 (padded) actions per block of SK waves, the waves splitting K.  No
// LDS staging: for MFMA s = 4t + q of its K range a lane supplies element q of
// a 16-byte load at k = 8t + 4 (lane / 32), for the weight row (lane % 32) and
// the env row (lane % 32) alike, so the two halves of the wave cover k = 8t ..
// 8t + 7 over four MFMAs.  A wave issues every load of its range before its
// first MFMA (one memory latency instead of one per K chunk).  The partial
// accumulators are added in LDS in wave order, then the sampling epilogue.
template <int MT, int SK>
__global__ __launch_bounds__(64 * SK) void sample_f32_splitk_kernel(GemmArgs g)
{
    constexpr int RED = (SK - 1) * MT * 16 * 64;
    constexpr int SO = 32 * 32 * MT;    // 32 envs x M_pad >= 32 x A floats
    constexpr int TCH = 16;             // 16-byte loads per operand row and chunk
    __shared__ __attribute__((aligned(16))) float lds[RED > SO ? RED : SO];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t n0 = (int64_t)blockIdx.x * 32;
    const int nt = g.K_pad / (8 * SK);  // 8-deep k groups per wave
    const int kb = wave * nt * 8;
    const int h = lane >> 5, r = lane & 31;
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.w, (short)0, (int)g.w_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.x, (short)0, (int)g.x_bytes, 0x00020000);
    // env rows past N lie past the extent and read as zero
    const uint32_t boff = (uint32_t)(((n0 + r) * g.ld_x + kb + 4 * h) * 4);
    uint32_t aoff[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) aoff[i] = (uint32_t)(((i * 32 + r) * g.K_pad + kb + 4 * h) * 4);

    f32x16_t acc[MT][1];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[i][0][q] = 0.0f;
    for (int t0 = 0; t0 < nt; t0 += TCH) {
        f32x4_t av[MT][TCH], bv[TCH];
        // past the wave's range the loads are skipped and their MFMAs add zero
#pragma unroll
        for (int u = 0; u < TCH; ++u) {
            const bool in = t0 + u < nt;
            const uint32_t dk = (uint32_t)(8 * (t0 + u) * 4);
            bv[u] = in ? __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(xr, boff + dk, 0, 0))
                       : f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int i = 0; i < MT; ++i)
                av[i][u] = in ? __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, aoff[i] + dk, 0, 0))
                              : f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        }
#pragma unroll
        for (int u = 0; u < TCH; ++u)
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][u][q], bv[u][q], acc[i][0], 0, 0, 0);
    }
    // partial sums: waves 1.. park theirs ([wave-1][i][reg][lane]), wave 0 adds
    // them in wave order
    if (wave > 0) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int q = 0; q < 16; ++q) lds[(((wave - 1) * MT + i) * 16 + q) * 64 + lane] = acc[i][0][q];
    }
    __syncthreads();
    if (wave == 0) {
        for (int w = 1; w < SK; ++w)
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int q = 0; q < 16; ++q) acc[i][0][q] += lds[(((w - 1) * MT + i) * 16 + q) * 64 + lane];
    }
    __syncthreads();
    // every wave joins the epilogue's barriers and wide stores; only wave 0's
    // columns are valid
    const int64_t nv = g.N - n0 < 32 ? g.N - n0 : 32;
    sample_epilogue<64 * SK, MT, 1>(g, lds, n0, nv, wave == 0 ? 0 : (1 << 20), tid, acc);
}

// ---------------------------------------------------------------------------
// bf16 layer GEMM for large batches.  Macro tile BM x BN (features x envs),
// K step BK; WM x WN waves, each owning a (BM/WM) x (BN/WN) block of 32x32
// MFMA tiles.  Two LDS stages: while the waves run the MFMAs of stage k from
// LDS, the 16-byte global loads of stage k+1 (issued one stage earlier) are
// written into the other LDS buffer and those of stage k+2 are issued.  Rows
// are padded by 16 bytes: at K step 64 (144-byte rows) the fragment reads
// and tile writes are free of bank conflicts (at K step 32, 80-byte rows, a
// third of the LDS cycles were conflicts).  Blocks are renumbered so that the
// feature blocks sharing one env block run on the same XCD (workgroups are
// dealt to the 8 XCDs round-robin) and share its L2.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, bool IN_OBS, bool SAMPLE>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_kernel(GemmArgs g)
{
    constexpr int NTHR = 64 * WM * WN;
    constexpr int KQ = BK / 8;                  // 16-byte chunks per row
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    constexpr int LDK = BK + 8;                 // bf16 elements per LDS row (144 bytes)
    constexpr int STAGE = (BM + BN) * LDK;      // elements per stage
    constexpr int A_CHUNKS = BM * KQ / NTHR;    // 16-byte chunks of the weight tile per thread
    static_assert(BM * KQ % NTHR == 0, "weight tile split");
    // activation tile: bf16 rows (hidden input) or fp32 observation rows
    constexpr int B_CHUNKS = BN * KQ / NTHR;    // hidden: 16-byte chunks per thread
    constexpr int B_TASKS = KQ * (BN / 4) / NTHR;  // obs: 8 k x 4 n blocks per thread
    static_assert(IN_OBS ? (KQ * (BN / 4) % NTHR == 0) : (BN * KQ % NTHR == 0), "split");

    // the epilogues reuse the stage buffers for the output tile (bf16 BM x BN,
    // or fp32 BN x A for the sampling layer)
    constexpr int OUT_ELEMS = SAMPLE ? 2 * BN * BM : BN * BM;
    constexpr int LDS_ELEMS = OUT_ELEMS > 2 * STAGE ? OUT_ELEMS : 2 * STAGE;
    __shared__ __attribute__((aligned(16))) uint16_t lds[LDS_ELEMS];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // XCD-aware renumbering of the 1-D grid
    const int mblocks = g.M_blocks;
    const int nblk = gridDim.x;
    int bid = blockIdx.x;
    if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
    const int64_t m0 = (int64_t)(bid % mblocks) * BM;
    const int64_t n0 = (int64_t)(bid / mblocks) * BN;

    const uint16_t *W = (const uint16_t *)g.w;
    const int nk = g.K_pad / BK;

    // Raw buffer descriptors: loads past num_records return zero, which pads
    // the env tail (rows n >= N) and the observation rows k >= D for free.
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.w, (short)0, (int)g.w_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.x, (short)0, (int)g.x_bytes, 0x00020000);

    u32x4_t ra[A_CHUNKS];
    u32x4_t rb[IN_OBS ? 1 : B_CHUNKS];
    f32x4_t ro[IN_OBS ? B_TASKS * 8 : 1];
    uint32_t a_off[A_CHUNKS], b_off[IN_OBS ? B_TASKS : B_CHUNKS];
#pragma unroll
    for (int c = 0; c < A_CHUNKS; ++c) {
        const int v = tid + c * NTHR;
        a_off[c] = (uint32_t)(((m0 + v / KQ) * g.K_pad + (v % KQ) * 8) * 2);
    }
    if constexpr (!IN_OBS) {
#pragma unroll
        for (int c = 0; c < B_CHUNKS; ++c) {
            const int v = tid + c * NTHR;
            b_off[c] = (uint32_t)(((n0 + v / KQ) * g.ld_x + (v % KQ) * 8) * 2);
        }
    } else {
#pragma unroll
        for (int t = 0; t < B_TASKS; ++t) {
            const int v = tid + t * NTHR;
            b_off[t] = (uint32_t)((((int64_t)(v % KQ) * 8) * g.ld_x + n0 + (v / KQ) * 4) * 4);
        }
    }

    auto load_global = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int c = 0; c < A_CHUNKS; ++c)
            ra[c] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, a_off[c], k0 * 2, 0));
        if constexpr (!IN_OBS) {
#pragma unroll
            for (int c = 0; c < B_CHUNKS; ++c)
                rb[c] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(xr, b_off[c], k0 * 2, 0));
        } else {
            const uint32_t row = (uint32_t)(g.ld_x * 4);
            const uint32_t kofs = (uint32_t)k0 * row;
#pragma unroll
            for (int t = 0; t < B_TASKS; ++t)
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    ro[t * 8 + j] = __builtin_bit_cast(
                        f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(xr, b_off[t] + j * row, kofs, 0));
        }
    };

    auto store_lds = [&](int buf) {
        uint16_t *As = lds + buf * STAGE;
        uint16_t *Bs = As + BM * LDK;
#pragma unroll
        for (int c = 0; c < A_CHUNKS; ++c) {
            const int v = tid + c * NTHR;
            const int r = v / KQ, q = v % KQ;
            *(u32x4_t *)(As + r * LDK + q * 8) = ra[c];
        }
        if constexpr (!IN_OBS) {
#pragma unroll
            for (int c = 0; c < B_CHUNKS; ++c) {
                const int v = tid + c * NTHR;
                const int r = v / KQ, q = v % KQ;
                *(u32x4_t *)(Bs + r * LDK + q * 8) = rb[c];
            }
        } else {
#pragma unroll
            for (int t = 0; t < B_TASKS; ++t) {
                const int v = tid + t * NTHR;
                const int kg = v % KQ, ng = v / KQ;
                const f32x4_t *o = ro + t * 8;
                // env ng*4+e gets the 8 consecutive k values kg*8..kg*8+7 (16 bytes)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    u32x4_t w;
                    w[0] = pack_bf16x2(o[0][e], o[1][e]);
                    w[1] = pack_bf16x2(o[2][e], o[3][e]);
                    w[2] = pack_bf16x2(o[4][e], o[5][e]);
                    w[3] = pack_bf16x2(o[6][e], o[7][e]);
                    *(u32x4_t *)(Bs + (ng * 4 + e) * LDK + kg * 8) = w;
                }
            }
        }
    };

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    auto compute = [&](int buf) {
        const uint16_t *As = lds + buf * STAGE;
        const uint16_t *Bs = As + BM * LDK;
        const int arow = wm * (TM * 32) + (lane & 31);
        const int brow = wn * (TN * 32) + (lane & 31);
        const int kof = 8 * (lane >> 5);
        constexpr int NS = BK / 16;
        bf16x8_t a[NS][TM], b[NS][TN];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[s][i] = *(const bf16x8_t *)(As + (arow + i * 32) * LDK + s * 16 + kof);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[s][j] = *(const bf16x8_t *)(Bs + (brow + j * 32) * LDK + s * 16 + kof);
        }
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s][i], b[s][j], acc[i][j], 0, 0, 0);
        // fragments of substep 0 first; the reads of each later substep are
        // spread over the MFMAs of the substep before it
        constexpr int F = TM + TN, MM = TM * TN;
        __builtin_amdgcn_sched_group_barrier(0x100, F, 0);
#pragma unroll
        for (int s = 0; s + 1 < NS; ++s)
#pragma unroll
            for (int x = 0; x < F; ++x) {
                __builtin_amdgcn_sched_group_barrier(0x008, (MM + F - 1) / F, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
        __builtin_amdgcn_sched_group_barrier(0x008, MM, 0);
    };

    load_global(0);
    store_lds(0);
    __syncthreads();
    if (nk > 1) load_global(1);
    for (int kt = 0; kt < nk; ++kt) {
        compute(kt & 1);
        if (kt + 1 < nk) store_lds((kt + 1) & 1);
        if (kt + 2 < nk) load_global(kt + 2);
        __syncthreads();
    }

    if constexpr (!SAMPLE) {
        // bias, ReLU, bf16; the tile is staged env-major in LDS ([env][feature]
        // rows of BM*2 bytes) and written out in whole rows.  A lane's four
        // features of one env are an 8-byte unit; units are XOR-swizzled by
        // env % (units per row), so that the 8-byte writes of 32 consecutive
        // envs hit distinct banks, and read back as 16-byte chunks (an odd
        // swizzle swaps the chunk's two halves, undone in registers).
        constexpr int CPR = BM / 8;             // 16-byte chunks per staged row
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int nl = wn * (TN * 32) + j * 32 + (lane & 31);
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) {
                    const int ml = wm * (TM * 32) + i * 32 + 8 * grp + 4 * (lane >> 5);
                    const float4 bb = *(const float4 *)(g.bias + m0 + ml);
                    const float v0 = fmaxf(acc[i][j][4 * grp + 0] + bb.x, 0.0f);
                    const float v1 = fmaxf(acc[i][j][4 * grp + 1] + bb.y, 0.0f);
                    const float v2 = fmaxf(acc[i][j][4 * grp + 2] + bb.z, 0.0f);
                    const float v3 = fmaxf(acc[i][j][4 * grp + 3] + bb.w, 0.0f);
                    const uint32_t lo = pack_bf16x2(v0, v1);
                    const uint32_t hi = pack_bf16x2(v2, v3);
                    const int unit = (ml >> 2) ^ (nl & (2 * CPR - 1));
                    *(uint2 *)(lds + nl * BM + unit * 4) = make_uint2(lo, hi);
                }
            }
        __syncthreads();
        uint16_t *Y = (uint16_t *)g.y;
        constexpr int RPP = NTHR / CPR;         // rows per pass
        const int cl = tid % CPR;
#pragma unroll 4
        for (int pass = 0; pass < BN / RPP; ++pass) {
            const int nl = pass * RPP + tid / CPR;
            const int64_t n = n0 + nl;
            const int sw = nl & (2 * CPR - 1);
            uint4 v = *(const uint4 *)(lds + nl * BM + ((cl ^ (sw >> 1)) * 8));
            if (sw & 1) v = make_uint4(v.z, v.w, v.x, v.y);
            if (n < g.N) *(uint4 *)(Y + n * g.ld_y + m0 + cl * 8) = v;
        }
    } else {
        // every action of an env lies in one wave (WM == 1, m0 == 0)
        const int64_t nv = g.N - n0 < BN ? g.N - n0 : BN;
        sample_epilogue<NTHR, TM, TN>(g, (float *)lds, n0, nv, wn * (TN * 32), tid, acc);
    }
}

template <int BM, int BN, int BK, int WM, int WN, bool IN_OBS, bool SAMPLE>
static hipError_t launch_bf16(GemmArgs g, int M_pad, hipStream_t s)
{
    g.M_blocks = M_pad / BM;
    const int64_t nb = (g.N + BN - 1) / BN;
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, BK, WM, WN, IN_OBS, SAMPLE>),
                       dim3((unsigned)(nb * g.M_blocks)), dim3(64 * WM * WN), 0, s, g);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// bf16 hidden-layer GEMM for large batches: persistent, ping-pong schedule.
// Tile 256x256 (features x envs), K step 64, 8 waves in two groups of four.
// Waves are dealt to the 4 SIMDs round-robin, so every SIMD holds one wave of
// each group.  Group g owns feature rows [128g, 128g+128) of a tile and its
// wave w env columns [64w, 64w+64): 4x2 MFMA tiles of 32x32 each.  The groups
// alternate between two phases separated by workgroup barriers: while one
// group runs the 32 MFMAs of a K step from fragments already in its
// registers, the other reads its fragments of the K step from LDS, so each
// SIMD's MFMA pipe is fed by one wave while the other waits on memory.
// Operands move global->LDS without passing through registers (buffer loads
// with the LDS flag, 16 bytes per lane; past the buffer end they return zero,
// which pads the env tail).  Issuing them holds up the issuing wave while the
// CU's memory pipeline drains (about 50 bytes per clock), so a K step's loads
// are split over its two phases: the reading group issues the activations
// (group 0) or its weight rows (group 1), and group 0 also issues its weight
// rows between its MFMAs.  A 128-byte LDS row holds its eight 16-byte chunks
// XOR-swizzled by (row/2)%8, so that fragment reads of 16 consecutive rows
// hit distinct banks.  Two LDS stages of 64 KB.
//
// One workgroup per CU walks a list of tiles, and the K steps of consecutive
// tiles form one pipeline: the next tile's first K step is loaded while the
// current one finishes.  A finished tile is written out (bias, ReLU, bf16) by
// both groups in the same phase, through a 2 KB LDS slot per wave, in
// 32-byte rows.  Tiles are ordered so that the workgroups of one XCD
// (workgroups are dealt to the 8 XCDs round-robin) share env blocks, whose
// activations then come from that XCD's L2.
// ---------------------------------------------------------------------------
#define IM_LDS_AS __attribute__((address_space(3)))

// s_waitcnt immediate that waits until at most n vector memory operations are
// outstanding (expcnt and lgkmcnt at their maxima)
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }
static_assert(vmcnt_imm(0) == 0x0F70 && vmcnt_imm(16) == 0x4F70, "s_waitcnt encoding");
__device__ __forceinline__ void wait_vmcnt0() { __builtin_amdgcn_s_waitcnt(vmcnt_imm(0)); }

// Global->LDS load of 16 bytes per lane, to LDS byte address lds + 16 * lane
// (lds wave-uniform), issued through inline assembly: the compiler then does
// not know that the instruction writes LDS, so it makes no later LDS access
// wait for it (it cannot tell the buffers apart, and would wait for every
// such load in flight); the kernel orders these loads itself with vmcnt waits
// and workgroup barriers.  m0, the instruction's LDS base, is restored; an
// SALU write of m0 needs one wait state before an LDS-DMA instruction reads
// it, which the compiler's hazard checks do not supply inside inline assembly.
__device__ __forceinline__ void lds_load16(__amdgpu_buffer_rsrc_t rsrc, uint32_t lds, uint32_t voff,
                                           uint32_t soff)
{
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\t"
                 "s_mov_b32 m0, %1\n\t"
                 "s_nop 0\n\t"
                 "buffer_load_dwordx4 %2, %3, %4 offen lds\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "s"(lds), "v"(voff), "s"(rsrc), "s"(soff)
                 : "memory");
}

// ReLU of a packed bf16 pair: a bf16 whose sign bit is set is a negative
// 16-bit integer, so a packed integer max with zero clears exactly the
// negative values (and -0).
typedef short im_s16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t relu_bf16x2(uint32_t p)
{
    const im_s16x2_t v = __builtin_bit_cast(im_s16x2_t, p);
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(v, (im_s16x2_t){0, 0}));
}

// LDS byte address of a __shared__ array
#define IM_LDS_ADDR(arr) ((uint32_t)(size_t)(IM_LDS_AS const void *)(arr))
__device__ __forceinline__ uint32_t uniform(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
__device__ __forceinline__ void wg_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__global__ __launch_bounds__(512) void gemm_bf16_pp_kernel(GemmArgs g)
{
    constexpr int BK = 64;
    constexpr int ROWB = BK * 2;                // bytes per LDS row
    constexpr int TILE_B = 256 * ROWB;          // one 256-row operand tile
    constexpr int STAGE_B = 2 * TILE_B;         // weight tile, then activation tile
    constexpr int EPI_B = 64 * 32;              // epilogue slot per wave: 64 envs x 16 features bf16
    constexpr int TM = 4, TN = 2, NS = BK / 16;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * STAGE_B];
    __shared__ __attribute__((aligned(16))) uint8_t epi_lds[8 * EPI_B];
    __shared__ __attribute__((aligned(16))) float bias_lds[2][256];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
    const int grp = wave >> 2, wi = wave & 3;

    // this workgroup's tiles: XCD x = blockIdx % 8 takes the x-th eighth of the
    // tile order (feature block fastest), its workgroups interleaved over it
    const int mblocks = g.M_blocks;
    const int64_t T = ((g.N + 255) / 256) * mblocks;
    const int per = (int)(gridDim.x >> 3);
    const int xcd = (int)(blockIdx.x & 7), slot = (int)(blockIdx.x >> 3);
    const int64_t r_begin = (xcd * T) / 8 + slot, r_end = ((xcd + 1) * T) / 8;
    if (slot >= per || r_begin >= r_end) return;
    const int n_tiles = (int)((r_end - r_begin + per - 1) / per);
    const int nk = g.K_pad / BK;
    const int S = n_tiles * nk;
    auto tile_m0 = [&](int ti) { return ((r_begin + (int64_t)ti * per) % mblocks) * 256; };
    auto tile_n0 = [&](int ti) { return ((r_begin + (int64_t)ti * per) / mblocks) * 256; };

    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.w, (short)0, (int)g.w_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.x, (short)0, (int)g.x_bytes, 0x00020000);

    // Loads: thread t of a group (t = tid % 256) fills 16-byte slot 256c + t of a
    // tile, c = 0..7: row 32c + t/8, physical chunk t%8, holding logical chunk
    // (t%8) ^ ((row/2)%8); the swizzle depends on t only.  The weight tile's rows
    // 0..127 (c = 0..3) are read only by group 0 and rows 128..255 (c = 4..7)
    // only by group 1, the activation tile by both.
    const int lrow = (tid & 255) >> 3;
    const int lq = (tid & 7) ^ ((lrow >> 1) & 7);
    const uint32_t a_voff = (uint32_t)((lrow * g.K_pad + lq * 8) * 2);
    const uint32_t b_voff = (uint32_t)((lrow * g.ld_x + lq * 8) * 2);
    const uint32_t lbase = IM_LDS_ADDR(lds) + (uint32_t)(((tid & 255) & ~63) * 16);
    // Activation row offsets stay in the per-lane offset (the part the buffer
    // range check sees), so rows past the env count read as zero; weight rows
    // are always in range.
    auto issue_x = [&](int st, int buf) {
        const int ti = st / nk, kt = st - ti * nk;
        const int64_t n0 = tile_n0(ti);
        const uint32_t base = lbase + (uint32_t)(buf * STAGE_B + TILE_B);
        const uint32_t k2 = uniform((uint32_t)(kt * BK * 2));
#pragma unroll
        for (int c = 0; c < 8; ++c)
            lds_load16(xr, uniform(base + c * 256 * 16),
                       b_voff + (uint32_t)(((n0 + 32 * c) * g.ld_x) * 2), k2);
    };
    // LDS address and buffer offset of the 32-row group c of the weight tile of
    // K step st (wave-uniform)
    auto w_lds = [&](int buf, int c) { return uniform(lbase + (uint32_t)(buf * STAGE_B + c * 256 * 16)); };
    auto w_off = [&](int st, int c) {
        const int ti = st / nk, kt = st - ti * nk;
        return uniform((uint32_t)(((tile_m0(ti) + 32 * c) * g.K_pad) * 2) + (uint32_t)(kt * BK * 2));
    };
    auto issue_w = [&](int st, int buf, int c) { lds_load16(wr, w_lds(buf, c), a_voff, w_off(st, c)); };

    // the 256 biases of tile ti into LDS buffer ti % 2, by one wave of group 1
    const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.bias, (short)0, (int)(g.M_blocks * 256 * 4), 0x00020000);
    auto stage_bias = [&](int ti) {
        lds_load16(br, uniform(IM_LDS_ADDR(bias_lds) + (uint32_t)((ti & 1) * 1024)), (uint32_t)(lane * 16),
                   uniform((uint32_t)(tile_m0(ti) * 4)));
    };

    bf16x8_t fa[NS][TM], fb[NS][TN];
    auto read_frags = [&](int buf) {
        const uint8_t *As = lds + buf * STAGE_B;
        const uint8_t *Bs = As + TILE_B;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int q = 2 * s + (lane >> 5);
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = grp * 128 + i * 32 + (lane & 31);
                fa[s][i] = *(const bf16x8_t *)(As + r * ROWB + ((q ^ ((r >> 1) & 7)) * 16));
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = wi * 64 + j * 32 + (lane & 31);
                fb[s][j] = *(const bf16x8_t *)(Bs + r * ROWB + ((q ^ ((r >> 1) & 7)) * 16));
            }
        }
        wait_lgkmcnt0();
    };

    f32x16_t acc[TM][TN];
    // A tile's accumulators start at the bias of their feature (row
    // 8 (r / 4) + 4 (lane / 32) + r % 4 of MFMA tile i holds feature
    // grp*128 + 32 i + that row), so the epilogue adds nothing.
    auto init_acc = [&](int ti) {
        const float *bias = bias_lds[ti & 1] + grp * 128 + 4 * (lane >> 5);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const f32x4_t b = *(const f32x4_t *)(bias + i * 32 + 8 * q);
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[i][j][4 * q + r] = b[r];
            }
    };
    auto mfma_sub = [&](int s) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s][j], acc[i][j], 0, 0, 0);
    };
    // The MFMAs of a K step.  With stw >= 0 (group 0), weight rows 0..127 of K
    // step stw are issued one 32-row group after each substep (addresses formed
    // before the first MFMA), so that the loads trickle into the memory pipeline
    // instead of holding up the MFMAs behind a queue of other loads.  One MFMA
    // sequence with wave-uniform branches: two copies of it exhaust the registers.
    auto mfma_step = [&](int stw, int bufw) {
        const bool ld = stw >= 0;
        uint32_t la[4] = {0, 0, 0, 0}, so[4] = {0, 0, 0, 0};
        if (ld) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                la[c] = w_lds(bufw, c);
                so[c] = w_off(stw, c);
            }
        }
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            mfma_sub(s);
            if (ld) lds_load16(wr, la[s], a_voff, so[s]);
        }
        __builtin_amdgcn_s_setprio(0);
    };

    // Writes this wave's 128x64 block of tile ti (ReLU, bf16; the accumulators
    // started at the bias) in eight passes of 16 features through its 2 KB slot
    // `ep`: [env][feature]
    // rows of 32 bytes, copied out 32 rows per wave instruction.  A lane's four
    // features of one env are an 8-byte unit, stored at unit (unit ^ s(env)),
    // s(env) = ((env >> 2) ^ (env >> 3)) % 4: the 8-byte writes of any 16 (and
    // of any 32) consecutive envs then hit distinct banks, and so do the 8-byte
    // reads of the copy-out (two per 16-byte store, since an odd s swaps a
    // chunk's two halves).  LDS operations of one wave complete in
    // order, so the slot needs no barrier between its writes and reads.
    // Issues exactly 16 buffer stores; rows past the env count get an offset
    // past the buffer end (the buffer range check drops such stores).
    //
    // The lane-dependent offsets are derived from an opaque copy of the lane
    // id: hoisted out of the K loop they would hold registers the loop needs.
    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
        g.y, (short)0, (int)g.y_bytes, 0x00020000);
    auto epilogue = [&](int ti, uint8_t *ep) {
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const uint32_t m0 = (uint32_t)tile_m0(ti), n0 = (uint32_t)tile_n0(ti);
        const uint32_t n_env = (uint32_t)g.N, ld_y = (uint32_t)g.ld_y;
        // the swizzle of env j*32 + ln%32 does not depend on j
        const int e = ln & 31;
        const int se = ((e >> 2) ^ (e >> 3)) & 3;
        uint8_t *wbase = ep + e * 32;
        const int rl = ln >> 1, c = ln & 1;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int hq = 0; hq < 2; ++hq) {
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    uint8_t *wj = wbase + j * 32 * 32;
#pragma unroll
                    for (int q2 = 0; q2 < 2; ++q2) {
                        const int q = 2 * hq + q2;
                        const uint32_t lo = relu_bf16x2(pack_bf16x2(acc[i][j][4 * q + 0], acc[i][j][4 * q + 1]));
                        const uint32_t hi = relu_bf16x2(pack_bf16x2(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]));
                        const int unit = (2 * q2 + (ln >> 5)) ^ se;
                        *(uint2 *)(wj + unit * 8) = make_uint2(lo, hi);
                    }
                }
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    // features 8c..8c+7 of the row: logical units 2c and 2c+1, at
                    // physical units (2c) ^ s and (2c+1) ^ s
                    const int row = p * 32 + rl;
                    const int sw = ((row >> 2) ^ (row >> 3)) & 3;
                    const uint8_t *rp = ep + row * 32 + ((c ^ (sw >> 1)) * 16);
                    const uint2 a = *(const uint2 *)(rp + (sw & 1) * 8);
                    const uint2 b = *(const uint2 *)(rp + ((sw & 1) ^ 1) * 8);
                    const u32x4_t v = {a.x, a.y, b.x, b.y};
                    // a row past the env count gets offset 0xFFFFFFF0 (all ones
                    // ORed in, no branch; offsets are multiples of 16), past every
                    // buffer the library accepts, with no dword of the store
                    // wrapping around 2^32
                    const uint32_t n = n0 + (uint32_t)(wi * 64 + row);
                    const uint32_t off =
                        (((n * ld_y + m0 + (uint32_t)(grp * 128 + i * 32 + hq * 16 + c * 8)) * 2u) |
                         (0u - (uint32_t)(n >= n_env))) & 0xFFFFFFF0u;
                    __builtin_amdgcn_raw_buffer_store_b128(v, yr, off, 0, 0);
                }
            }
        }
    };

    // Phase 2st: group 0 reads K step st and loads the activations of st+1 into
    // the other buffer (last read by group 1 in phase 2st-1).  Phase 2st+1: group
    // 0 runs the MFMAs of st and, between them, loads weight rows 0..127 of st+2
    // into the buffer it has just read (only group 0 reads those rows); group 1
    // reads st and loads weight rows 128..255 of st+1 (its own rows, last read
    // in phase 2st-1).  Each phase thus carries half a K step's operand bytes,
    // and every load has two phases or more to land.  Loads of a wave complete
    // in issue order: group 0 waits at the end of phase 2st+1 for all but the 4
    // loads of st+2, group 1 at the end of phase 2st+2 for all of its loads.
    if (grp == 0) {
        issue_x(0, 0);
#pragma unroll
        for (int c = 0; c < 4; ++c) issue_w(0, 0, c);
        if (S > 1) {
#pragma unroll
            for (int c = 0; c < 4; ++c) issue_w(1, 1, c);
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(4));
        } else {
            wait_vmcnt0();
        }
    } else {
        if (wi == 0) stage_bias(0);
#pragma unroll
        for (int c = 4; c < 8; ++c) issue_w(0, 0, c);
        wait_vmcnt0();
    }
    wg_barrier();
    init_acc(0);
    if (grp == 1) wg_barrier();
    uint8_t *my_ep = epi_lds + wave * EPI_B;
    for (int st = 0; st < S; ++st) {
        const int buf = st & 1;
        const int kt = st % nk, ti = st / nk;
        // Group 0 writes a finished tile at the start of the tile's next read
        // phase, group 1 right after the tile's last MFMAs: the same phase, so
        // that the MFMA pipes stand idle through one epilogue per tile, not two.
        if (grp == 0 && st > 0 && kt == 0) {
            epilogue(ti - 1, my_ep);
            init_acc(ti);
        }
        // group 1, in a tile's first K step: the next tile's biases (the
        // buffer's previous biases were read when the tile before started)
        if (grp == 0) {
            if (st + 1 < S) issue_x(st + 1, buf ^ 1);
        } else {
            if (wi == 0 && kt == 0 && ti + 1 < n_tiles) stage_bias(ti + 1);
            if (st + 1 < S) {
#pragma unroll
                for (int c = 4; c < 8; ++c) issue_w(st + 1, buf ^ 1, c);
            }
        }
        read_frags(buf);
        wg_barrier();
        const bool wt = grp == 0 && st + 2 < S;
        mfma_step(wt ? st + 2 : -1, buf);
        if (wt) __builtin_amdgcn_s_waitcnt(vmcnt_imm(4));
        else wait_vmcnt0();
        if (grp == 1 && kt == nk - 1) {
            epilogue(ti, my_ep);
            if (ti + 1 < n_tiles) init_acc(ti + 1);
        }
        wg_barrier();
    }
    if (grp == 0) {
        wg_barrier();
        epilogue(n_tiles - 1, my_ep);
    }
}

static hipError_t launch_bf16_pp(GemmArgs g, int M_pad, hipStream_t s)
{
    g.M_blocks = M_pad / 256;
    g.y_bytes = (uint32_t)((uint64_t)g.N * (uint64_t)g.ld_y * 2);
    const int64_t tiles = ((g.N + 255) / 256) * g.M_blocks;
    int P = g.n_cu > 0 ? (g.n_cu & ~7) : 256;
    if (P < 8) P = 8;
    // fewer tiles than CUs: one tile per workgroup
    if (tiles < P) P = (int)((tiles + 7) & ~7);
    hipLaunchKernelGGL(gemm_bf16_pp_kernel, dim3((unsigned)P), dim3(512), 0, s, g);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Observation staging for the first bf16 layer of a large batch: obs fp32
// [D][ld] (env fastest) -> bf16 [N][K_pad] (feature fastest, zero for
// features >= D), rounded to nearest even exactly as the GEMM's own
// observation path rounds.  Block: 64 envs; per 64-feature chunk the block
// reads 64 rows of 64 envs (16-byte loads along envs), transposes through LDS
// (65-float rows: conflict-free column reads) and writes 128-byte feature
// runs per env.  The ping-pong GEMM then streams the staged copy like any
// hidden layer.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void stage_obs_bf16_kernel(const float *__restrict__ obs, int64_t ld,
                                                             int D, int64_t N, int K_pad,
                                                             uint32_t obs_bytes, uint16_t *__restrict__ x16)
{
    __shared__ float t[64][65];
    const int tid = threadIdx.x;
    const int64_t n0 = (int64_t)blockIdx.x * 64;
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        (void *)obs, (short)0, (int)obs_bytes, 0x00020000);
    const bool vec = ((ld & 3) == 0) && ((((uintptr_t)obs) & 15) == 0);
    for (int k0 = 0; k0 < K_pad; k0 += 64) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int idx = tid + 256 * i;
            const int row = idx >> 4, q = idx & 15;
            const int f = k0 + row;
            // features >= D lie past the buffer extent and read as zero
            const uint32_t off = (uint32_t)(((int64_t)f * ld + n0 + 4 * q) * 4);
            f32x4_t v;
            if (vec) {
                v = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off + 4 * e, 0, 0));
            }
            if (f >= D) v = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int e = 0; e < 4; ++e) t[row][4 * q + e] = v[e];
        }
        __syncthreads();
        const int nl = tid >> 2, r0 = (tid & 3) * 16;
        const int64_t n = n0 + nl;
        if (n < N) {
            uint32_t w[8];
#pragma unroll
            for (int h = 0; h < 8; ++h)
                w[h] = pack_bf16x2(t[r0 + 2 * h][nl], t[r0 + 2 * h + 1][nl]);
            uint4 *dst = (uint4 *)(x16 + n * K_pad + k0 + r0);
            dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
            dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// The whole bf16 policy in one kernel.  One workgroup of 8 waves per 64 envs
// runs every layer; between layers the activations stay in LDS as [64 envs][K]
// bf16 rows whose 16-byte chunks (8 features) are XOR-swizzled by env % 16,
// so that the fragment reads and the output writes of 16 consecutive envs
// hit distinct banks.  No activation goes through memory; the LDS (about
// 136 KB) holds one workgroup per CU, and a batch larger than 64 envs per CU
// runs in successive rounds of workgroups.
//
// Hidden layer of width M: wave w owns output features [w M/8, (w+1) M/8),
// M/256 MFMA tiles of 32 rows, for all 64 envs (2 tiles of 32).  Its weight
// fragments (A operand) come from global memory straight into registers,
// loaded one K step (64) ahead: every workgroup reads the same weights (a
// copy in MFMA fragment order), which stay in the L2, so each weight byte
// from the L2 serves 64 envs (128 flop).  The env fragments (B operand) are
// read from LDS.  The accumulators start at the bias; once every wave has
// read the layer's input (workgroup barrier) they are written over it: ReLU,
// bf16, and the two half waves trade four-feature groups so that each lane
// stores whole 16-byte chunks.  The last layer and the sampling use every
// wave (fused_last).
// ---------------------------------------------------------------------------
constexpr int FUSED_BN = 64;                      // envs per workgroup
constexpr int FUSED_ROW = FUSED_MAX_WIDTH * 2;    // LDS bytes per env

// LDS byte offset of 16-byte chunk c of env e in rows of rs bytes
__device__ __forceinline__ uint32_t fused_off(int e, int c, int rs)
{
    return (uint32_t)(e * rs + ((c ^ (e & 15)) << 4));
}

// The observation [D][ld] fp32 into the first layer's LDS rows as bf16, by
// K step (64 features, eight 16-byte chunks: one per wave); lane = env, so
// that each load instruction reads 64 consecutive envs of one feature.  The
// feature's row offset is wave-uniform (a scalar offset); features past D go
// through a descriptor of extent zero and read as zero; lanes past the last
// env read env 0 (every address stays inside the buffer, whether or not the
// descriptor's range check counts the scalar offset) and are zeroed by store().
struct ObsStream {
    __amdgpu_buffer_rsrc_t r, r0;
    int64_t ld;
    uint32_t nb;     // this lane's env, in bytes (0 past the last env)
    int D, wave, lane, rs;
    bool nvalid;
    __device__ __forceinline__ void load(int ks, float (&v)[8]) const
    {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int k = 64 * ks + 8 * wave + i;
            const bool in = k < D;
            v[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                 in ? r : r0, nb, in ? (int)((int64_t)k * ld * 4) : 0, 0));
        }
    }
    __device__ __forceinline__ void store(uint8_t *act, int ks, const float (&v)[8]) const
    {
        float x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = nvalid ? v[i] : 0.0f;
        *(u32x4_t *)(act + fused_off(lane, 8 * ks + wave, rs)) =
            u32x4_t{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                    pack_bf16x2(x[6], x[7])};
    }
};

// acc[TM][TN] += W[rows][K] X[envs][K]^T: rows w_row0 + 32 mt + lane % 32 of
// the weights (w in fragment order, frag_index), envs e0 + 32 nt + lane % 32
// of the LDS rows (rs bytes each).  MFMA substep s of K step ks takes
// k = 64 ks + 16 s + 8 (lane / 32) .. +7 for both operands; its weight
// fragment is one 1 KB block, 16 consecutive bytes per lane (in the weights'
// row-major layout a wavefront's 16-byte pieces would lie in 32 rows, and the
// vector L1 serves such a load at a fraction of the rate of whole lines).
// The weight loads of K step ks + 1 are issued right after the MFMAs of the
// same substep of step ks (held there by scheduling barriers: the compiler
// would otherwise gather them at the end of the step); in the last step they
// go through a descriptor of extent zero, which makes them return zero
// without a memory access (a branch around them would make the compiler copy
// the fragments).  The env fragments of the next substep are read from LDS
// before the MFMAs of the current one.
template <int TM, int TN, bool DRAIN>
__device__ __forceinline__ void fused_mma(const uint16_t *w, uint32_t w_bytes, int w_row0, int nks,
                                          int ks0, int ks1, const uint8_t *act, int rs, int e0,
                                          int lane, f32x16_t (&acc)[TM][TN])
{
    const int r = lane & 31, h = lane >> 5;
    if (ks0 >= ks1) return;
    const __amdgpu_buffer_rsrc_t wr =
        __builtin_amdgcn_make_buffer_rsrc((void *)w, (short)0, (int)w_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t wr0 = __builtin_amdgcn_make_buffer_rsrc((void *)w, (short)0, 0, 0x00020000);
    // byte offset of this lane's 16 bytes in a fragment block (a vector
    // offset) and of tile mt's K step ks (a scalar offset)
    const uint32_t vo = (uint32_t)(16 * lane);
    int so[TM];
#pragma unroll
    for (int mt = 0; mt < TM; ++mt) so[mt] = (w_row0 / 32 + mt) * nks * 4096;
    // the caller's loads that the loop uses (the biases the accumulators
    // start from) complete here, so that no wait for them lands inside it
    if (DRAIN) __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __builtin_amdgcn_sched_barrier(0);
    // in the order of the loop's own loads, which its waits count on
    u32x4_t wa[TM][4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int mt = 0; mt < TM; ++mt)
            wa[mt][s] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                        wr, vo + 1024 * s, so[mt] + ks0 * 4096, 0));
        __builtin_amdgcn_sched_barrier(0);
    }
    bf16x8_t bn[TN];
#pragma unroll
    for (int nt = 0; nt < TN; ++nt)
        bn[nt] = *(const bf16x8_t *)(act + fused_off(e0 + 32 * nt + r, 8 * ks0 + h, rs));
    for (int ks = ks0; ks < ks1; ++ks) {
        const bool more = ks + 1 < ks1;
        const __amdgpu_buffer_rsrc_t wk = more ? wr : wr0;
        const int kn = (ks + 1) * 4096;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            bf16x8_t b[TN];
#pragma unroll
            for (int nt = 0; nt < TN; ++nt) b[nt] = bn[nt];
            // next substep's chunk (the last step re-reads its own chunk 0)
            const int cn = s < 3 ? 8 * ks + 2 * (s + 1) + h : (more ? 8 * (ks + 1) + h : 8 * ks + h);
#pragma unroll
            for (int nt = 0; nt < TN; ++nt)
                bn[nt] = *(const bf16x8_t *)(act + fused_off(e0 + 32 * nt + r, cn, rs));
#pragma unroll
            for (int mt = 0; mt < TM; ++mt)
#pragma unroll
                for (int nt = 0; nt < TN; ++nt)
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8_t, wa[mt][s]), b[nt], acc[mt][nt], 0, 0, 0);
#pragma unroll
            for (int mt = 0; mt < TM; ++mt)
                wa[mt][s] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                            wk, vo + 1024 * s, so[mt] + kn, 0));
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// Hidden layer l of width M = 256 TM: LDS rows of rs bytes in, M * 2 out.
template <int TM>
__device__ __forceinline__ void fused_hidden(const FusedMlpArgs &f, int l, uint8_t *act, int rs,
                                             int wave, int lane)
{
    const int K = f.K_pad[l], h = lane >> 5, r = lane & 31;
    const int fm = wave * TM * 32;
    f32x16_t acc[TM][2];
#pragma unroll
    for (int mt = 0; mt < TM; ++mt)
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
            const float4 bb = *(const float4 *)(f.bias[l] + fm + mt * 32 + 8 * grp + 4 * h);
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {
                acc[mt][nt][4 * grp + 0] = bb.x;
                acc[mt][nt][4 * grp + 1] = bb.y;
                acc[mt][nt][4 * grp + 2] = bb.z;
                acc[mt][nt][4 * grp + 3] = bb.w;
            }
        }
    fused_mma<TM, 2, true>(f.w[l], f.w_bytes[l], fm, K / 64, 0, K / 64, act, rs, 0, lane, acc);
    __syncthreads();
    const int rso = 2 * TM * 256;
#pragma unroll
    for (int mt = 0; mt < TM; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            uint32_t p[4][2];
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                p[grp][0] = relu_bf16x2(pack_bf16x2(acc[mt][nt][4 * grp + 0], acc[mt][nt][4 * grp + 1]));
                p[grp][1] = relu_bf16x2(pack_bf16x2(acc[mt][nt][4 * grp + 2], acc[mt][nt][4 * grp + 3]));
            }
            // 16-byte chunk j (features 8j .. 8j+7 of the tile) is group j of
            // both half waves: lanes of half 0 keep chunks 0 and 2, half 1
            // chunks 1 and 3.  v_permlane32_swap exchanges the upper half-wave
            // of its first operand with the lower half of its second, so
            // after swapping (group 0, group 1) every lane holds its chunk
            // as (first, second), likewise (group 2, group 3)
            const auto a0 = __builtin_amdgcn_permlane32_swap(p[0][0], p[1][0], false, false);
            const auto a1 = __builtin_amdgcn_permlane32_swap(p[0][1], p[1][1], false, false);
            const auto b0 = __builtin_amdgcn_permlane32_swap(p[2][0], p[3][0], false, false);
            const auto b1 = __builtin_amdgcn_permlane32_swap(p[2][1], p[3][1], false, false);
            const u32x4_t ca = u32x4_t{a0[0], a1[0], a0[1], a1[1]};
            const u32x4_t cb = u32x4_t{b0[0], b1[0], b0[1], b1[1]};
            const int e = 32 * nt + r, c = (fm + 32 * mt) / 8 + h;
            *(u32x4_t *)(act + fused_off(e, c, rso)) = ca;
            *(u32x4_t *)(act + fused_off(e, c + 2, rso)) = cb;
        }
    __syncthreads();
}

// Last layer and sampling.  The 32 MT padded actions of the 64 envs are 2 MT
// MFMA tiles of 32 x 32.  Up to MT = 3 a wave takes one action tile for both
// env halves over one of KS = 8 / MT slices of K (two at MT = 3), so that
// each slice of the weights is loaded once per workgroup; at MT = 4, where
// those partial tiles would not fit in LDS next to the mean and action rows,
// a wave takes one (tile, env half) over the whole of K.  Every wave but two
// at MT = 3 has work.  The partial tiles go to LDS and all 512 threads then take one
// (env, block of four actions) at a time: the mean is the bias plus the
// partials in slice order, the noise comes from Philox, action = mean +
// sigma z, and each env's logp adds its blocks' sums in block order.  log
// sigma, the biases and the envs' step counters are loaded before the
// layer's MFMAs and staged in LDS after them.
template <int MT>
__device__ __forceinline__ void fused_last(const FusedMlpArgs &f, uint8_t *act, int rs, int64_t n0,
                                           int64_t nv, int wave, int tid)
{
    constexpr int TN = MT == 4 ? 1 : 2;                       // env halves per wave
    constexpr int KS = MT == 4 ? 1 : (MT == 3 ? 2 : 8 / MT);  // K slices
    constexpr int MP = 32 * MT;
    // partial tiles, mean and action rows and the per-block sums over the input rows
    static_assert((KS * FUSED_BN * MP + 2 * FUSED_BN * MP + FUSED_BN * 33) * 4 <= FUSED_BN * FUSED_ROW,
                  "last-layer LDS");
    const GemmArgs &g = f.out;
    const int l = f.L - 1, nks = f.K_pad[l] / 64, lane = tid & 63, A = g.A;
    __shared__ float sig[128], sbias[128], slp0;
    __shared__ uint32_t senv[FUSED_BN];
    float p0 = 0.0f, p1 = 0.0f;
    uint32_t en = 0;
    if (wave == 0) {
        if (lane < A) p0 = g.log_std[lane];
        if (lane + 64 < A) p1 = g.log_std[lane + 64];
    } else if (wave == 1) {
        if (lane < A) p0 = g.bias[lane];
        if (lane + 64 < A) p1 = g.bias[lane + 64];
    } else if (wave == 2 && lane < nv) {
        en = g.env_n[n0 + lane];
    }
    f32x16_t acc[1][TN];
#pragma unroll
    for (int nt = 0; nt < TN; ++nt)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[0][nt][q] = 0.0f;
    // wave -> (env half when TN = 1, action tile, K slice)
    const int nt0 = TN == 1 ? (wave & 1) : 0;
    const int wt = TN == 1 ? (wave >> 1) : wave;
    const int mt = wt % MT, ksl = wt / MT;
    const bool active = wave < (2 / TN) * MT * KS;
    if (active)
        fused_mma<1, TN, false>(f.w[l], f.w_bytes[l], 32 * mt, nks, ksl * nks / KS,
                                (ksl + 1) * nks / KS, act, rs, 32 * nt0, lane, acc);
    __syncthreads();
    // the layer input is read: partial tiles [KS][64 envs][MP] fp32 (16-byte
    // units XOR-swizzled by env % 8), mean and action rows [64][A], and the
    // per-block sums of z^2 / 2 [64][33] take its place
    float *part = (float *)act;
    float *smean = part + KS * FUSED_BN * MP;
    float *sact = smean + FUSED_BN * A;
    float *slp = sact + FUSED_BN * A;
    if (active) {
#pragma unroll
        for (int nt = 0; nt < TN; ++nt) {
            const int e = 32 * (nt0 + nt) + (lane & 31), h = lane >> 5;
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const int unit = (8 * mt + 2 * grp + h) ^ (e & 7);
                *(f32x4_t *)(part + (ksl * FUSED_BN + e) * MP + 4 * unit) =
                    f32x4_t{acc[0][nt][4 * grp], acc[0][nt][4 * grp + 1], acc[0][nt][4 * grp + 2],
                            acc[0][nt][4 * grp + 3]};
            }
        }
    }
    if (wave == 0) {
        if (lane < A) sig[lane] = expf(p0);
        if (lane + 64 < A) sig[lane + 64] = expf(p1);
        float c = (lane < A ? p0 + HALF_LOG_2PI : 0.0f) + (lane + 64 < A ? p1 + HALF_LOG_2PI : 0.0f);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
        if (lane == 0) slp0 = c;
    } else if (wave == 1) {
        if (lane < A) sbias[lane] = p0;
        if (lane + 64 < A) sbias[lane + 64] = p1;
    } else if (wave == 2) {
        senv[lane] = en;
    }
    __syncthreads();
    const int G = (A + 3) / 4;
    for (int it = tid; it < FUSED_BN * G; it += 512) {
        const int e = it & (FUSED_BN - 1), j = it / FUSED_BN;
        if (e >= nv) continue;
        float mu[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) mu[q] = 4 * j + q < A ? sbias[4 * j + q] : 0.0f;
#pragma unroll
        for (int k = 0; k < KS; ++k) {
            const f32x4_t v = *(const f32x4_t *)(part + (k * FUSED_BN + e) * MP + 4 * (j ^ (e & 7)));
#pragma unroll
            for (int q = 0; q < 4; ++q) mu[q] += v[q];
        }
        float z[4];
        normals4(g.seed, (uint32_t)(n0 + e), senv[e], (uint32_t)j, 0u, z);
        float lp = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int m = 4 * j + q;
            if (m < A) {
                smean[e * A + m] = mu[q];
                sact[e * A + m] = mu[q] + sig[m] * z[q];
                lp += 0.5f * z[q] * z[q];
            }
        }
        slp[e * 33 + j] = lp;
    }
    __syncthreads();
    if (tid < nv && g.logp) {
        float sum = 0.0f;
        for (int j = 0; j < G; ++j) sum += slp[tid * 33 + j];
        g.logp[n0 + tid] = -(sum + slp0);
    }
    copy_rows_out<512>(g.mean + n0 * A, smean, nv * A, tid);
    copy_rows_out<512>(g.action + n0 * A, sact, nv * A, tid);
}

// The critic's output: v = head . h + bias over the last hidden layer's
// activations h (bf16 in LDS, rows of rs bytes) with the fp32 head.  Wave w
// sums chunks [w C/8, (w+1) C/8) of every env (lane), the eight partial sums
// are added in wave order.
__device__ __forceinline__ void fused_value_head(const FusedMlpArgs &f, const uint8_t *act, int rs,
                                                 int64_t n0, int64_t nv, int wave, int tid)
{
    __shared__ float spart[8][FUSED_BN];
    const int K = f.M_pad[f.L - 1], per = K / 64, e = tid & (FUSED_BN - 1);
    float acc = 0.0f;
    for (int j = 0; j < per; ++j) {
        const int c = wave * per + j;
        const u32x4_t v = *(const u32x4_t *)(act + fused_off(e, c, rs));
        const float *w = f.head + 8 * c;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            acc += w[2 * q] * __uint_as_float(v[q] << 16);
            acc += w[2 * q + 1] * __uint_as_float(v[q] & 0xFFFF0000u);
        }
    }
    spart[wave][e] = acc;
    __syncthreads();
    if (tid < nv) {
        float sum = f.head[K];
#pragma unroll
        for (int p = 0; p < 8; ++p) sum += spart[p][tid];
        f.value[n0 + tid] = sum;
    }
}

// The whole observation of the block staged before the first layer: every
// load (up to S K steps, one chunk each per wave) is issued before the first
// is written, one memory latency in all.
template <int S>
__device__ __forceinline__ void fused_stage_obs(const ObsStream &os, uint8_t *act, int nks)
{
    float v[S][8];
#pragma unroll
    for (int j = 0; j < S; ++j)
        if (j < nks) os.load(j, v[j]);
#pragma unroll
    for (int j = 0; j < S; ++j)
        if (j < nks) os.store(act, j, v[j]);
}

// VALUE: a critic (every layer hidden, then the value head).
template <bool VALUE>
__global__ __launch_bounds__(512) void policy_fused_bf16_kernel(FusedMlpArgs f)
{
    __shared__ __attribute__((aligned(16))) uint8_t act[FUSED_BN * FUSED_ROW];
    const int tid = threadIdx.x, lane = tid & 63, wave = (int)uniform((uint32_t)tid >> 6);
    const int64_t n0 = (int64_t)blockIdx.x * FUSED_BN;
    const int64_t nv = f.out.N - n0 < FUSED_BN ? f.out.N - n0 : FUSED_BN;

    // observation [D][ld] fp32 -> bf16 rows of 16-byte chunks (8 features)
    int rs = ((f.K_pad[0] + 127) & ~127) * 2;
    ObsStream os;
    os.r = __builtin_amdgcn_make_buffer_rsrc((void *)f.obs, (short)0, (int)f.obs_bytes, 0x00020000);
    os.r0 = __builtin_amdgcn_make_buffer_rsrc((void *)f.obs, (short)0, 0, 0x00020000);
    os.ld = f.ld_obs;
    os.nb = lane < nv ? (uint32_t)((n0 + lane) * 4) : 0u;
    os.D = f.D;
    os.wave = wave;
    os.lane = lane;
    os.rs = rs;
    os.nvalid = lane < nv;
    const int nks0 = f.K_pad[0] / 64;
    if (nks0 <= 4) fused_stage_obs<4>(os, act, nks0);
    else if (nks0 <= 8) fused_stage_obs<8>(os, act, nks0);
    else fused_stage_obs<16>(os, act, nks0);
    __syncthreads();
    for (int l = 0; l + (VALUE ? 0 : 1) < f.L; ++l) {
        switch (f.M_pad[l] >> 8) {
            case 1: fused_hidden<1>(f, l, act, rs, wave, lane); break;
            case 2: fused_hidden<2>(f, l, act, rs, wave, lane); break;
            case 3: fused_hidden<3>(f, l, act, rs, wave, lane); break;
            default: fused_hidden<4>(f, l, act, rs, wave, lane); break;
        }
        rs = 2 * f.M_pad[l];
    }
    if constexpr (VALUE) {
        fused_value_head(f, act, rs, n0, nv, wave, tid);
        return;
    }
    switch (f.M_pad[f.L - 1] >> 5) {
        case 1: fused_last<1>(f, act, rs, n0, nv, wave, tid); break;
        case 2: fused_last<2>(f, act, rs, n0, nv, wave, tid); break;
        case 3: fused_last<3>(f, act, rs, n0, nv, wave, tid); break;
        default: fused_last<4>(f, act, rs, n0, nv, wave, tid); break;
    }
}

// Shapes the kernel assumes; n_hidden: the layers that are hidden.
static bool fused_shapes_ok(const FusedMlpArgs &f, int n_hidden)
{
    if (f.L < 1 || f.L > FUSED_MAX_LAYERS || f.K_pad[0] > FUSED_MAX_WIDTH || (f.K_pad[0] & 63) ||
        f.K_pad[0] <= 0)
        return false;
    for (int l = 0; l < f.L; ++l) {
        if (l > 0 && f.K_pad[l] != f.M_pad[l - 1]) return false;
        if (l < n_hidden && (f.M_pad[l] > FUSED_MAX_WIDTH || (f.M_pad[l] & 255) || f.M_pad[l] <= 0))
            return false;
    }
    return true;
}

hipError_t launch_policy_fused(const FusedMlpArgs &f, hipStream_t s)
{
    if (f.out.N <= 0) return hipSuccess;
    if (!fused_shapes_ok(f, f.L - 1) || f.M_pad[f.L - 1] > 128 || (f.M_pad[f.L - 1] & 31) ||
        f.M_pad[f.L - 1] <= 0 || f.out.A > f.M_pad[f.L - 1])
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(policy_fused_bf16_kernel<false>,
                       dim3((unsigned)((f.out.N + FUSED_BN - 1) / FUSED_BN)), dim3(512), 0, s, f);
    return hipGetLastError();
}

hipError_t launch_value_fused(const FusedMlpArgs &f, hipStream_t s)
{
    if (f.out.N <= 0) return hipSuccess;
    if (!fused_shapes_ok(f, f.L) || !f.head || !f.value) return hipErrorInvalidValue;
    hipLaunchKernelGGL(policy_fused_bf16_kernel<true>,
                       dim3((unsigned)((f.out.N + FUSED_BN - 1) / FUSED_BN)), dim3(512), 0, s, f);
    return hipGetLastError();
}

template <bool IN_OBS, int BN, int WN>
static hipError_t launch_bf16_sample_t(const GemmArgs &g, int M_pad, hipStream_t s)
{
    switch (M_pad / 32) {
        case 1: return launch_bf16<32, BN, 64, 1, WN, IN_OBS, true>(g, M_pad, s);
        case 2: return launch_bf16<64, BN, 64, 1, WN, IN_OBS, true>(g, M_pad, s);
        case 3: return launch_bf16<96, BN, 64, 1, WN, IN_OBS, true>(g, M_pad, s);
        default: return launch_bf16<128, BN, 64, 1, WN, IN_OBS, true>(g, M_pad, s);
    }
}

template <bool IN_OBS>
static hipError_t launch_bf16_sample(const GemmArgs &g, int M_pad, hipStream_t s)
{
    if (g.N <= SMALL_BATCH) return launch_bf16_sample_t<IN_OBS, 64, 2>(g, M_pad, s);
    return launch_bf16_sample_t<IN_OBS, 128, 4>(g, M_pad, s);
}

// fp32 layers: 128x128 tiles (2x2 waves of 64x64) for large batches; for
// small batches 64x64 tiles (one 32x32 MFMA tile per wave) so that a layer
// still spreads over every SIMD.

template <bool BF16, bool IN_OBS, int MT, int NT>
static hipError_t launch_hidden_t(const GemmArgs &g, int M_pad, hipStream_t s)
{
    constexpr int WGM = 2, WGN = 2;
    const dim3 grid((unsigned)(M_pad / (WGM * MT * 32)),
                    (unsigned)((g.N + WGN * NT * 32 - 1) / (WGN * NT * 32)));
    static_assert(!BF16, "bf16 layers use gemm_bf16_kernel");
    hipLaunchKernelGGL((gemm_f32_kernel<IN_OBS, false, WGM, WGN, MT, NT>), grid,
                       dim3(64 * WGM * WGN), 0, s, g);
    return hipGetLastError();
}

template <bool BF16, bool IN_OBS>
static hipError_t launch_hidden(const GemmArgs &g, int M_pad, hipStream_t s)
{
    if (g.N <= SMALL_BATCH) return launch_hidden_t<BF16, IN_OBS, 1, 1>(g, M_pad, s);
    return launch_hidden_t<BF16, IN_OBS, 2, 2>(g, M_pad, s);
}

template <bool BF16, bool IN_OBS, int MT, int WGN>
static hipError_t launch_sample_t(const GemmArgs &g, hipStream_t s)
{
    const dim3 grid(1u, (unsigned)((g.N + WGN * 32 - 1) / (WGN * 32)));
    static_assert(!BF16, "bf16 layers use gemm_bf16_kernel");
    hipLaunchKernelGGL((gemm_f32_kernel<IN_OBS, true, 1, WGN, MT, 1>), grid,
                       dim3(64 * WGN), 0, s, g);
    return hipGetLastError();
}

template <bool BF16, bool IN_OBS, int MT>
static hipError_t launch_sample_mt(const GemmArgs &g, hipStream_t s)
{
    if (g.N <= SMALL_BATCH) return launch_sample_t<BF16, IN_OBS, MT, 1>(g, s);
    return launch_sample_t<BF16, IN_OBS, MT, 4>(g, s);
}

template <int MT>
static hipError_t launch_sample_splitk(const GemmArgs &g, hipStream_t s)
{
    hipLaunchKernelGGL((sample_f32_splitk_kernel<MT, 4>), dim3((unsigned)((g.N + 31) / 32)),
                       dim3(256), 0, s, g);
    return hipGetLastError();
}

template <bool BF16, bool IN_OBS>
static hipError_t launch_sample(const GemmArgs &g, int M_pad, hipStream_t s)
{
    // small batches, hidden input (K_pad a multiple of 32: 8-deep groups per wave)
    if (!IN_OBS && g.N <= SMALL_BATCH && (g.K_pad & 31) == 0) {
        switch (M_pad / 32) {
            case 1: return launch_sample_splitk<1>(g, s);
            case 2: return launch_sample_splitk<2>(g, s);
            case 3: return launch_sample_splitk<3>(g, s);
            default: return launch_sample_splitk<4>(g, s);
        }
    }
    switch (M_pad / 32) {
        case 1: return launch_sample_mt<BF16, IN_OBS, 1>(g, s);
        case 2: return launch_sample_mt<BF16, IN_OBS, 2>(g, s);
        case 3: return launch_sample_mt<BF16, IN_OBS, 3>(g, s);
        default: return launch_sample_mt<BF16, IN_OBS, 4>(g, s);
    }
}

// Host entry used by the C ABI layer: one layer.
hipError_t launch_policy_layer(bool bf16, bool in_obs, bool sample, const GemmArgs &g, int M_pad,
                               hipStream_t s, bool *staged)
{
    if (g.N <= 0) return hipSuccess;
    if (bf16) {
        // large batches: the ping-pong kernel (256x256 tiles of 8 waves, K step
        // 64) on bf16 hidden inputs, and on the observation once staged as bf16
        // [N][K_pad]; the last layer 128 envs per block of 4 waves
        if (!sample) {
            if (g.N <= SMALL_BATCH)
                return in_obs ? launch_bf16<128, 128, 64, 2, 2, true, false>(g, M_pad, s)
                              : launch_bf16<128, 128, 64, 2, 2, false, false>(g, M_pad, s);
            // the ping-pong kernel needs whole 256-feature blocks and >= 2 K steps
            const bool pp = (M_pad & 255) == 0 && (g.K_pad & 63) == 0 && g.K_pad >= 128;
            if (!in_obs && pp) return launch_bf16_pp(g, M_pad, s);
            if (!in_obs) return launch_bf16<256, 256, 64, 2, 4, false, false>(g, M_pad, s);
            if (!g.x16 || !pp)
                return launch_bf16<256, 256, 64, 2, 4, true, false>(g, M_pad, s);
            if (!g.x16_staged) {
                hipLaunchKernelGGL(stage_obs_bf16_kernel, dim3((unsigned)((g.N + 63) / 64)), dim3(256),
                                   0, s, (const float *)g.x, g.ld_x, g.K_valid, g.N, g.K_pad,
                                   g.x_bytes, (uint16_t *)g.x16);
                hipError_t e = hipGetLastError();
                if (e != hipSuccess) return e;
            }
            if (staged) *staged = true;
            GemmArgs h = g;
            h.x = g.x16;
            h.ld_x = g.K_pad;
            h.x_bytes = (uint32_t)((uint64_t)g.N * (uint64_t)g.K_pad * 2);
            return launch_bf16_pp(h, M_pad, s);
        }
        return in_obs ? launch_bf16_sample<true>(g, M_pad, s) : launch_bf16_sample<false>(g, M_pad, s);
    }
    if (!sample)
        return in_obs ? launch_hidden<false, true>(g, M_pad, s) : launch_hidden<false, false>(g, M_pad, s);
    return in_obs ? launch_sample<false, true>(g, M_pad, s) : launch_sample<false, false>(g, M_pad, s);
}

}  // namespace im
