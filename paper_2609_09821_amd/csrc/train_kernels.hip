// train_kernels.hip -- the PPO update (the training loop's update_policy of
// Fig. 3) for bf16 actor-critic MLPs: minibatch gather from the rollout
// storage, forward and backward GEMMs on MFMA, the clipped-surrogate loss,
// deterministic gradient reductions, global-norm clip, KL-adaptive learning
// rate and Adam, all on the device with no host round trip.
//
// Layout: every activation and gradient is feature-major, [features][Mb]
// with the minibatch's samples contiguous (bf16), so the MFMA accumulator
// (one sample per lane, four consecutive features per register group) is
// stored without a transpose, and all three products of a layer
//   forward  Y^T  = W   X^T          (out x Mb)
//   backward dX^T = W^T dZ^T         (in x Mb, masked by the ReLU)
//   weights  dW   = dZ^T X           (out x in, reduced over the minibatch)
// run on one GEMM kernel C[m][n] = sum_k A[m][k] B(k, n): A always has k
// contiguous (weights, transposed weights, dZ^T), B either k-major [k][n]
// (activations, gradients) or n-major [n][k] (X^T for the weight gradient).
#include <hip/hip_runtime.h>

#include "device_math.h"
#include "launch.h"

namespace im {

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4_v __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_v __attribute__((ext_vector_type(2)));
typedef short v4s_t __attribute__((ext_vector_type(4)));
#define IM_LDS3 __attribute__((address_space(3)))

// Sum of x over each group of W (16 or 32) consecutive lanes, aligned to W,
// returned in the group's last lane: an inclusive scan within each 16-lane
// row (DPP row shifts by 1, 2, 4, 8; lanes shifted in from outside the row
// read zero), then for W = 32 the total of the even row added into the odd
// row (row broadcast of lane 15).  The order of the additions is fixed.
// x plus the value DPP control CTRL brings in (0 where it brings none: lanes
// outside ROW_MASK, or shifted in from outside the row).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float x)
{
    const int t = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROW_MASK, 0xF, true);
    return x + __builtin_bit_cast(float, t);
}

template <int W>
__device__ __forceinline__ float lane_group_sum(float x)
{
    static_assert(W == 16 || W == 32, "lane group");
    x = dpp_add<0x111, 0xF>(x);     // row_shr:1
    x = dpp_add<0x112, 0xF>(x);     // row_shr:2
    x = dpp_add<0x114, 0xF>(x);     // row_shr:4
    x = dpp_add<0x118, 0xF>(x);     // row_shr:8
    if constexpr (W == 32)
        x = dpp_add<0x142, 0xA>(x); // row_bcast:15 into rows 1 and 3 (row mask 0b1010)
    return x;
}

// ---------------------------------------------------------------------------
// GEMM: tiles of BM = 64 WM rows by BN columns (WM x 2 waves, each wave
// 64 x BN/2 = 2 x BN/64 MFMA 32x32x16 tiles).  launch_tgemm picks WM = 4
// (256 rows, 8 waves, 512 threads) when M is a multiple of 256, else WM = 2
// (128 rows, 4 waves), and BN = 256 when N is a multiple of 256, else 128:
// 256 x 256 tiles of 8 waves wherever the shape allows.  K step 64, two LDS
// stages; loads of stage k+2 are in flight while stage k runs.  k-contiguous
// operands sit in LDS rows of 72 bf16 (144 bytes: fragment reads free of bank
// conflicts).  A k-major B tile is stored as it lies in memory, [64 k][BN n]
// in rows of BN + 16 bf16, and its
// MFMA fragments are read with the LDS transpose read: in every 16-lane
// group, lane 4j+q addresses row k0+j, columns n0+4q..n0+4q+3, and lane l
// receives rows k0..k0+3 of column n0+l (two reads give the 8 consecutive k
// of a bf16 fragment; the 32-byte row shift of the padding keeps a group's
// four rows on distinct banks).  blockIdx.y splits K (weight gradients: K =
// the minibatch).  All operands are zero-padded to whole tiles.
// ---------------------------------------------------------------------------
template <bool BT, int EPI, int WM, int BN>
__global__ __launch_bounds__(128 * WM) void tgemm_kernel(TGemm g)
{
    // WM x 2 waves, each 64 x BN/2 (TN = BN/64 MFMA tiles across); tile BM x BN
    constexpr int NT = 128 * WM;
    constexpr int TN = BN / 64;
    constexpr int BM = 64 * WM, BK = 64, LDK = BK + 8;
    constexpr int LDN = BN + 16;                // k-major B rows (bf16)
    static_assert(BK * LDN <= BN * LDK + BK * 16, "stage size");
    constexpr int STAGE = BM * LDK + (BT ? BK * LDN : BN * LDK);
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;   // wave: 64 x 64 of the tile
    const int mblocks = g.M / BM;
    const int64_t m0 = (int64_t)(blockIdx.x % mblocks) * BM;
    const int64_t n0 = (int64_t)(blockIdx.x / mblocks) * BN;
    const int kb = blockIdx.y * g.k_split;
    const int ke = kb + g.k_split < g.K ? kb + g.k_split : g.K;
    const int nk = (ke - kb) / BK;
    // mask bits (256x256 tiles): the 16 pieces this thread writes in the
    // epilogue, one byte of 8 samples each, 16 contiguous bytes per thread
    constexpr bool MBITS = BM == 256 && BN == 256 && (EPI == T_HIDDEN || EPI == T_MASK);
    uint4 mbits_in = make_uint4(0u, 0u, 0u, 0u);
    if constexpr (MBITS && EPI == T_MASK)
        if (g.mbits) mbits_in = g.mbits[(int64_t)blockIdx.x * NT + tid];

    const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.A, (short)0, (int)g.a_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g.B, (short)0, (int)g.b_bytes, 0x00020000);

    // A: BM rows x 8 chunks of 16 bytes; B: BN rows x 8 chunks (n-major) or
    // 64 rows x BN/8 chunks of 8 samples (k-major)
    constexpr int AC = BM * 8 / NT, BC = BN * 8 / NT;
    constexpr int BQ = BN / 8;                  // k-major chunks per row
    uint32_t a_off[AC], b_off[BC];
#pragma unroll
    for (int c = 0; c < AC; ++c) {
        const int v = tid + c * NT;
        a_off[c] = (uint32_t)(((m0 + (v >> 3)) * g.lda + kb + (v & 7) * 8) * 2);
    }
#pragma unroll
    for (int c = 0; c < BC; ++c) {
        const int v = tid + c * NT;
        if constexpr (!BT) b_off[c] = (uint32_t)(((n0 + (v >> 3)) * g.ldb + kb + (v & 7) * 8) * 2);
        else b_off[c] = (uint32_t)((((int64_t)kb + v / BQ) * g.ldb + n0 + (v % BQ) * 8) * 2);
    }
    const uint32_t bt_row = (uint32_t)(g.ldb * 2);

    u32x4_v ra[AC], rb[BC];
    auto load_global = [&](int kt) {
        const int kofs = kt * BK;
#pragma unroll
        for (int c = 0; c < AC; ++c)
            ra[c] = __builtin_bit_cast(u32x4_v, __builtin_amdgcn_raw_buffer_load_b128(ar, a_off[c], kofs * 2, 0));
        const uint32_t s = BT ? (uint32_t)kofs * bt_row : (uint32_t)kofs * 2;
#pragma unroll
        for (int c = 0; c < BC; ++c)
            rb[c] = __builtin_bit_cast(u32x4_v, __builtin_amdgcn_raw_buffer_load_b128(br, b_off[c], s, 0));
    };
    auto store_lds = [&](int buf) {
        uint16_t *As = lds + buf * STAGE;
        uint16_t *Bs = As + BM * LDK;
#pragma unroll
        for (int c = 0; c < AC; ++c) {
            const int v = tid + c * NT;
            *(u32x4_v *)(As + (v >> 3) * LDK + (v & 7) * 8) = ra[c];
        }
#pragma unroll
        for (int c = 0; c < BC; ++c) {
            const int v = tid + c * NT;
            if constexpr (!BT) *(u32x4_v *)(Bs + (v >> 3) * LDK + (v & 7) * 8) = rb[c];
            else *(u32x4_v *)(Bs + (v / BQ) * LDN + (v % BQ) * 8) = rb[c];
        }
    };

    f32x16_t acc[2][TN];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // transpose-read addressing of the k-major B fragments (see above):
    // 16-lane group gi covers columns 16 (gi & 1).. and k rows 8 (gi >> 1)..
    const int gi = lane >> 4, si = lane & 15;
    static_assert(BM * (BN + 8) <= 2 * STAGE, "epilogue tile fits the stages");
    const int tr_off = (8 * (gi >> 1) + (si >> 2)) * LDN + 16 * (gi & 1) + 4 * (si & 3);
    auto compute = [&](int buf) {
        const uint16_t *As = lds + buf * STAGE;
        const uint16_t *Bs = As + BM * LDK;
        const int arow = wm * 64 + (lane & 31);
        const int brow = wn * (BN / 2) + (lane & 31);
        const int kof = 8 * (lane >> 5);
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            bf16x8_t a[2], b[TN];
#pragma unroll
            for (int i = 0; i < 2; ++i) a[i] = *(const bf16x8_t *)(As + (arow + i * 32) * LDK + s * 16 + kof);
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                if constexpr (!BT) {
                    b[j] = *(const bf16x8_t *)(Bs + (brow + j * 32) * LDK + s * 16 + kof);
                } else {
                    const uint16_t *p = Bs + (s * 16) * LDN + wn * (BN / 2) + j * 32 + tr_off;
                    const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((IM_LDS3 v4s_t *)p);
                    const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((IM_LDS3 v4s_t *)(p + 4 * LDN));
                    const short v8[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                    b[j] = __builtin_bit_cast(bf16x8_t, v8);
                }
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    };

    if (nk > 0) {
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
    }

    // epilogue: lane (l & 31) holds sample column n, registers 4*grp + q the
    // rows 8*grp + 4*(l >> 5) + q of each 32 x 32 tile
    if constexpr (EPI == T_HIDDEN || EPI == T_MASK) {
        // bf16 tile staged in LDS as [m][n] (rows of BN + 8), then written in
        // 16-byte row pieces; the ReLU mask is read the same way
        constexpr int LDO = BN + 8;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int nl = wn * (BN / 2) + j * 32 + (lane & 31);
#pragma unroll
                for (int grp = 0; grp < 4; ++grp)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int ml = wm * 64 + i * 32 + 8 * grp + 4 * (lane >> 5) + q;
                        float v = acc[i][j][4 * grp + q];
                        if constexpr (EPI == T_HIDDEN) v = fmaxf(v + g.bias[m0 + ml], 0.0f);
                        lds[ml * LDO + nl] = f32_to_bf16_rne(v);
                    }
            }
        __syncthreads();
        // BM rows x BN/8 pieces of 8 samples
        uint32_t mbits_out[4] = {0u, 0u, 0u, 0u};
        const uint32_t mbits_w[4] = {mbits_in.x, mbits_in.y, mbits_in.z, mbits_in.w};
#pragma unroll
        for (int c = 0; c < BM * BQ / NT; ++c) {
            const int v = tid + c * NT;
            const int ml = v / BQ, pc = v % BQ;
            uint4 o = *(const uint4 *)(lds + ml * LDO + pc * 8);
            const int64_t off = (m0 + ml) * g.ldc + n0 + pc * 8;
            if constexpr (MBITS && EPI == T_HIDDEN) {
                // bit 2k (2k+1) of the piece's byte: the low (high) half of word k is > 0
                const uint32_t ow[4] = {o.x, o.y, o.z, o.w};
                uint32_t byte = 0u;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t lo = ow[k] & 0xFFFFu, hi = ow[k] >> 16;
                    byte |= ((lo != 0 && !(lo & 0x8000u)) ? 1u : 0u) << (2 * k);
                    byte |= ((hi != 0 && !(hi & 0x8000u)) ? 1u : 0u) << (2 * k + 1);
                }
                mbits_out[c >> 2] |= byte << (8 * (c & 3));
            }
            if constexpr (EPI == T_MASK) {
                uint32_t ow[4] = {o.x, o.y, o.z, o.w};
                if (MBITS && g.mbits) {
                    const uint32_t byte = (mbits_w[c >> 2] >> (8 * (c & 3))) & 0xFFu;
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        ow[k] &= ((byte >> (2 * k)) & 1u ? 0x0000FFFFu : 0u) |
                                 ((byte >> (2 * k + 1)) & 1u ? 0xFFFF0000u : 0u);
                } else {
                    const uint4 h = *(const uint4 *)(g.mask + (m0 + ml) * g.ldm + n0 + pc * 8);
                    const uint32_t hw[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        // keep each half where the activation (bf16) is > 0
                        const uint32_t lo = hw[k] & 0xFFFFu, hi = hw[k] >> 16;
                        const uint32_t keep = ((lo != 0 && !(lo & 0x8000u)) ? 0x0000FFFFu : 0u) |
                                              ((hi != 0 && !(hi & 0x8000u)) ? 0xFFFF0000u : 0u);
                        ow[k] &= keep;
                    }
                }
                o = make_uint4(ow[0], ow[1], ow[2], ow[3]);
                if (g.rs_part) {
                    // the row's sum over this tile's columns: the BQ consecutive lanes
                    // holding the row's pieces are summed by a fixed DPP pattern into
                    // the group's last lane
                    float rs = 0.0f;
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        rs += bf16_to_f32((uint16_t)(ow[k] & 0xFFFFu)) + bf16_to_f32((uint16_t)(ow[k] >> 16));
                    rs = lane_group_sum<BQ>(rs);
                    if (pc == BQ - 1) g.rs_part[(m0 + ml) * (g.N / BN) + n0 / BN] = (double)rs;
                }
            }
            *(uint4 *)((uint16_t *)g.C + off) = o;
        }
        if constexpr (MBITS && EPI == T_HIDDEN)
            if (g.mbits)
                g.mbits[(int64_t)blockIdx.x * NT + tid] =
                    make_uint4(mbits_out[0], mbits_out[1], mbits_out[2], mbits_out[3]);
    } else {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int64_t n = n0 + wn * (BN / 2) + j * 32 + (lane & 31);
#pragma unroll
                for (int grp = 0; grp < 4; ++grp)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int64_t m = m0 + wm * 64 + i * 32 + 8 * grp + 4 * (lane >> 5) + q;
                        const float v = acc[i][j][4 * grp + q];
                        if constexpr (EPI == T_LINEAR) {
                            if (m < g.M_valid) ((float *)g.C)[m * g.ldc + n] = v + g.bias[m];
                        } else {
                            ((float *)g.C)[((int64_t)blockIdx.y * g.M + m) * g.ldc + n] = v;
                        }
                    }
            }
    }
}

// ---------------------------------------------------------------------------
// Minibatch gather.  Column j = 64 c + l of the minibatch is env e0 + l of
// step t, where chunk c of the minibatch is q = perm[c]: t = q / (N/64),
// e0 = 64 (q % (N/64)).  One wavefront per chunk; chunks past the
// minibatch's end write zeros (padding columns).  The chunk's actions and
// means ([64][A] floats, contiguous in the [T][N][A] storage) are read 32
// columns at a time with loads of whole 128-byte row pieces into the wave's
// LDS slice (rows of 33 floats: the transposed reads hit 64 distinct banks)
// and written out as [A][Mb] rows of 64 samples.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a)
{
    constexpr int KC = 32, LDC = KC + 1;
    __shared__ float gather_lds[4][64 * LDC];
    const int lane = threadIdx.x & 63;
    const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
    float *sh = gather_lds[threadIdx.x >> 6];
    if (c >= a.chunks_pad) return;
    const int64_t j = (int64_t)c * 64 + lane;
    const int64_t Mb = a.Mb_pad;
    if (c >= a.chunks) {
        for (int i = 0; i < a.K0; ++i) a.x0[i * Mb + j] = 0;
        for (int k = 0; k < a.A; ++k) {
            a.act[k * Mb + j] = 0.0f;
            a.mean_old[k * Mb + j] = 0.0f;
        }
        a.logp_old[j] = 0.0f;
        a.adv[j] = 0.0f;
        a.ret[j] = 0.0f;
        a.vold[j] = 0.0f;
        return;
    }
    int q = a.perm[c];
    q = q < 0 ? 0 : (q >= a.n_chunks ? a.n_chunks - 1 : q);   // memory safety only
    const int64_t t = q / a.cpt;
    const int64_t e = (int64_t)(q % a.cpt) * 64 + lane;
    const float *o = a.obs + t * a.D * a.ld + e;
    int i = 0;
    for (; i + 8 <= a.D; i += 8) {
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = o[(int64_t)(i + k) * a.ld];
#pragma unroll
        for (int k = 0; k < 8; ++k) a.x0[(i + k) * Mb + j] = f32_to_bf16_rne(v[k]);
    }
    for (; i < a.D; ++i) a.x0[i * Mb + j] = f32_to_bf16_rne(o[(int64_t)i * a.ld]);
    for (; i < a.K0; ++i) a.x0[i * Mb + j] = 0;
    const int64_t blk = (t * a.N + (e - lane)) * a.A;   // the chunk's [64][A] block
#pragma unroll 1
    for (int arr = 0; arr < 2; ++arr) {
        const float *src = (arr == 0 ? a.action : a.mean) + blk;
        float *dst = arr == 0 ? a.act : a.mean_old;
        for (int k0 = 0; k0 < a.A; k0 += KC) {
            const int kc = a.A - k0 < KC ? a.A - k0 : KC;
            // the LDS slice is the wave's own and a wave's LDS operations complete
            // in order: no barrier between these writes and the reads below
#pragma unroll 4
            for (int x = lane; x < 64 * KC; x += 64) {
                const int r = x / KC, cc = x % KC;
                if (cc < kc) sh[r * LDC + cc] = src[(int64_t)r * a.A + k0 + cc];
            }
            for (int cc = 0; cc < kc; ++cc) dst[(int64_t)(k0 + cc) * Mb + j] = sh[lane * LDC + cc];
        }
    }
    const int64_t s = t * a.ld + e;
    a.logp_old[j] = a.logp[s];
    a.adv[j] = a.adv_src[s];
    a.ret[j] = a.ret_src[s];
    a.vold[j] = a.value[s];
}

// ---------------------------------------------------------------------------
// Critic head (width-1 output layer) on feature-major activations.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void head_forward_kernel(const uint16_t *__restrict__ h, int K,
                                                           int64_t Mb, const float *__restrict__ w,
                                                           const float *__restrict__ b,
                                                           float *__restrict__ v)
{
    // 8 consecutive samples per thread (16-byte loads); each sample's sum runs
    // over k in order, as one sample per thread would
    const int64_t j = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
    if (j >= Mb) return;
    float acc[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
    for (int k = 0; k < K; ++k) {
        const uint4 x = *(const uint4 *)(h + k * Mb + j);
        const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
        const float wk = w[k];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            acc[2 * q] += wk * bf16_to_f32((uint16_t)(xw[q] & 0xFFFFu));
            acc[2 * q + 1] += wk * bf16_to_f32((uint16_t)(xw[q] >> 16));
        }
    }
    const float4 o0 = make_float4(acc[0] + b[0], acc[1] + b[0], acc[2] + b[0], acc[3] + b[0]);
    const float4 o1 = make_float4(acc[4] + b[0], acc[5] + b[0], acc[6] + b[0], acc[7] + b[0]);
    *(float4 *)(v + j) = o0;
    *(float4 *)(v + j + 4) = o1;
}

// dZ^T[k][j] = w[k] dV[j] where h[k][j] > 0 (bf16), for the last hidden
// layer; rows K..gridDim.y-1 (padding) are zero.  8 samples per thread.
// Optionally the block's float64 partial sums of row k < K, at
// [k][blockIdx.x]: pw of h[k][j] dV[j] (the head's weight gradient), pb of
// the stored dZ^T[k][j] (the layer's bias gradient); each thread's 8 terms in
// order, a fixed wavefront butterfly, the 4 wave sums in wave order.
__global__ __launch_bounds__(256) void head_backward_kernel(const uint16_t *__restrict__ h, int K,
                                                            int64_t Mb,
                                                            const float *__restrict__ w,
                                                            const float *__restrict__ dv,
                                                            uint16_t *__restrict__ dz,
                                                            double *__restrict__ pw,
                                                            double *__restrict__ pb)
{
    __shared__ double red[2][4];
    const int64_t j = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
    const int k = blockIdx.y;
    double sw = 0.0, sb = 0.0;
    if (j < Mb) {
        uint4 *out = (uint4 *)(dz + k * Mb + j);
        if (k >= K) {
            *out = make_uint4(0u, 0u, 0u, 0u);
        } else {
            const uint4 x = *(const uint4 *)(h + k * Mb + j);
            const float4 d0 = *(const float4 *)(dv + j), d1 = *(const float4 *)(dv + j + 4);
            const float d[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
            const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
            const float wk = w[k];
            uint32_t o[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t lo = xw[q] & 0xFFFFu, hi = xw[q] >> 16;
                const uint32_t a = (lo != 0 && !(lo & 0x8000u)) ? f32_to_bf16_rne(wk * d[2 * q]) : 0u;
                const uint32_t b = (hi != 0 && !(hi & 0x8000u)) ? f32_to_bf16_rne(wk * d[2 * q + 1]) : 0u;
                o[q] = a | (b << 16);
                sw += (double)bf16_to_f32((uint16_t)lo) * (double)d[2 * q];
                sw += (double)bf16_to_f32((uint16_t)hi) * (double)d[2 * q + 1];
                sb += (double)bf16_to_f32((uint16_t)a);
                sb += (double)bf16_to_f32((uint16_t)b);
            }
            *out = make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
    if (k >= K || (!pw && !pb)) return;     // uniform over the block
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        sw += __shfl_xor(sw, o);
        sb += __shfl_xor(sb, o);
    }
    if (lane == 0) {
        red[0][wave] = sw;
        red[1][wave] = sb;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        const double t = ((red[threadIdx.x][0] + red[threadIdx.x][1]) + red[threadIdx.x][2]) +
                         red[threadIdx.x][3];
        double *p = threadIdx.x == 0 ? pw : pb;
        if (p) p[(int64_t)k * gridDim.x + blockIdx.x] = t;
    }
}

// ---------------------------------------------------------------------------
// Per-row sums over the minibatch, float64 in a fixed order:
// out[r] = sum_j x[r][j] (x bf16 or fp32), optionally times y[j].  Each row
// is cut into `parts` segments (blockIdx.y), read in 16-byte pieces; the
// segment sums are added in segment order by rowsum_finish_kernel.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ __launch_bounds__(256) void rowsum_kernel(const void *__restrict__ x, int64_t Mb,
                                                     const float *__restrict__ y, int parts,
                                                     double *__restrict__ part)
{
    __shared__ double red[256];
    constexpr int E = BF16 ? 8 : 4;             // elements per 16-byte piece
    const int r = blockIdx.x, seg = blockIdx.y;
    const int64_t len = Mb / parts;             // Mb and len are multiples of 256
    const int64_t j0 = seg * len;
    double s = 0.0;
    for (int64_t j = j0 + (int64_t)threadIdx.x * E; j < j0 + len; j += 256 * E) {
        float v[E];
        if constexpr (BF16) {
            const uint4 q = *(const uint4 *)((const uint16_t *)x + r * Mb + j);
            const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v[2 * k] = bf16_to_f32((uint16_t)(w[k] & 0xFFFF));
                v[2 * k + 1] = bf16_to_f32((uint16_t)(w[k] >> 16));
            }
        } else {
            const float4 q = *(const float4 *)((const float *)x + r * Mb + j);
            v[0] = q.x;
            v[1] = q.y;
            v[2] = q.z;
            v[3] = q.w;
        }
        if (y) {
#pragma unroll
            for (int k = 0; k < E; ++k) s += (double)v[k] * (double)y[j + k];
        } else {
#pragma unroll
            for (int k = 0; k < E; ++k) s += (double)v[k];
        }
    }
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) part[(int64_t)r * parts + seg] = red[0];
}

// One block per row: thread i adds parts i, i + 256, ... in order, then a
// fixed tree over the block.
__global__ __launch_bounds__(256) void rowsum_finish_rows_kernel(const double *__restrict__ part,
                                                                 int parts, float *__restrict__ out)
{
    __shared__ double red[256];
    const int r = blockIdx.x;
    double s = 0.0;
    for (int k = threadIdx.x; k < parts; k += 256) s += part[(int64_t)r * parts + k];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[r] = (float)red[0];
}

__global__ __launch_bounds__(256) void rowsum_finish_kernel(const double *__restrict__ part, int rows,
                                                            int parts, float *__restrict__ out)
{
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= rows) return;
    double s = 0.0;
    for (int k = 0; k < parts; ++k) s += part[(int64_t)r * parts + k];
    out[r] = (float)s;
}

// Weight gradient from the split-K partials: out[o][i] = sum_z P[z][o][i]
// (z in order) for o < rows, i < cols.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float *__restrict__ P, int S,
                                                            int64_t M, int64_t N, int rows,
                                                            int cols, float *__restrict__ out)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)rows * cols) return;
    const int64_t o = idx / cols, i = idx % cols;
    float s = 0.0f;
    for (int z = 0; z < S; ++z) s += P[((int64_t)z * M + o) * N + i];
    out[idx] = s;
}

// ---------------------------------------------------------------------------
// Loss: per sample, the clipped surrogate, value loss and KL; writes the
// bf16 output-layer gradient dmu^T [A][Mb] (zero for padding columns), dV,
// and per-block float64 partials: the log-std gradient (A) then the stats.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void loss_kernel(LossArgs a)
{
    __shared__ double red[4][MAX_ACTIONS + LOSS_STATS];
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t Mb = a.Mb_pad;
    const bool live = j < a.Mb;
    const double n = (double)a.n_samples;
    const double amean = a.summary[IM_SUM_ADVANTAGE] / n;
    const double avar = (a.summary[IM_SUM_ADVANTAGE_SQ] - a.summary[IM_SUM_ADVANTAGE] * amean) / (n - 1.0);
    const double astd = sqrt(avar > 0.0 ? avar : 0.0);
    const float inv_mb = 1.0f / (float)a.Mb;
    float g_logp = 0.0f, l_pi = 0.0f, l_v = 0.0f, kl = 0.0f, clipped = 0.0f;
    float logp = 0.0f, ratio = 1.0f;
    if (live) {
        for (int k = 0; k < a.A; ++k) {
            const float ls = a.log_std[k];
            const float sig = expf(ls);
            const float d = a.act[k * Mb + j] - a.mean[k * Mb + j];
            logp -= d * d / (2.0f * sig * sig) + ls + 0.91893853320467274f;
        }
        ratio = expf(logp - a.logp_old[j]);
        const float A = (float)(((double)a.adv[j] - amean) / (astd + 1e-8));
        const float rc = fminf(fmaxf(ratio, 1.0f - a.clip), 1.0f + a.clip);
        const float s1 = -A * ratio, s2 = -A * rc;
        l_pi = fmaxf(s1, s2);
        g_logp = (s1 >= s2 ? -A * ratio : 0.0f) * inv_mb;
        clipped = fabsf(ratio - 1.0f) > a.clip ? 1.0f : 0.0f;
        // value loss
        const float V = a.value[j], R = a.ret[j], Vo = a.vold[j];
        float dv;
        if (a.clipped_value_loss) {
            const float dvo = V - Vo;
            const float Vc = Vo + fminf(fmaxf(dvo, -a.clip), a.clip);
            const float e1 = (V - R) * (V - R), e2 = (Vc - R) * (Vc - R);
            l_v = fmaxf(e1, e2);
            const bool inside = dvo > -a.clip && dvo < a.clip;
            dv = e1 >= e2 ? 2.0f * (V - R) : (inside ? 2.0f * (Vc - R) : 0.0f);
        } else {
            l_v = (V - R) * (V - R);
            dv = 2.0f * (V - R);
        }
        a.dv[j] = a.value_coef * dv * inv_mb;
        for (int k = 0; k < a.A; ++k) {
            const float ls = a.log_std[k], lso = a.log_std_old[k];
            const float sig2 = expf(2.0f * ls), so2 = expf(2.0f * lso);
            const float dm = a.mean_old[k * Mb + j] - a.mean[k * Mb + j];
            kl += ls - lso + (so2 + dm * dm) / (2.0f * sig2) - 0.5f;
        }
    } else if (j < Mb) {
        a.dv[j] = 0.0f;
    }
    // Per action: the mean's gradient (bf16) and the block partial of the
    // log-std gradient; then the four stats.  Each partial is summed over a
    // wavefront by a fixed butterfly, and the block's four wave sums are added
    // in wave order.
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    auto wave_sum = [](double x) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
        return x;
    };
    for (int k = 0; k < a.A; ++k) {
        float gm = 0.0f;
        double x = 0.0;
        if (live) {
            const float sig2 = expf(2.0f * a.log_std[k]);
            const float d = a.act[k * Mb + j] - a.mean[k * Mb + j];
            gm = g_logp * d / sig2;
            x = (double)g_logp * ((double)d * d / sig2 - 1.0);
        }
        if (j < Mb) a.dmu[k * Mb + j] = f32_to_bf16_rne(gm);
        x = wave_sum(x);
        if (lane == 0) red[wave][k] = x;
    }
    const float st[LOSS_STATS] = {l_pi, l_v, kl, clipped};
#pragma unroll
    for (int q = 0; q < LOSS_STATS; ++q) {
        const double x = wave_sum(live ? (double)st[q] : 0.0);
        if (lane == 0) red[wave][a.A + q] = x;
    }
    __syncthreads();
    const int nf = a.A + LOSS_STATS;
    for (int f = threadIdx.x; f < nf; f += 256)
        a.partial[(int64_t)blockIdx.x * nf + f] = ((red[0][f] + red[1][f]) + red[2][f]) + red[3][f];
}

// ---------------------------------------------------------------------------
// Optimizer.  norm_kernel: per-block float64 sums of g^2 over the flat
// gradient.  finalize_kernel (one block): the minibatch's log-std gradient
// (loss partials + entropy term) into the flat gradient, the loss stats,
// the global norm and clip factor, the KL-adaptive learning rate, the Adam
// step count and bias corrections.  adam_kernel: the step.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void norm_kernel(const float *__restrict__ g, int64_t P,
                                                   double *__restrict__ partial)
{
    __shared__ double red[256];
    double s = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < P; i += (int64_t)gridDim.x * 256)
        s += (double)g[i] * (double)g[i];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[blockIdx.x] = red[0];
}

// the log-std gradient and loss stats of the minibatch from the loss
// partials: one block per field, a fixed tree over the blocks' partials
__global__ __launch_bounds__(256) void loss_reduce_kernel(LossReduceArgs r)
{
    __shared__ double red[256];
    const int nf = r.A + LOSS_STATS;
    const int f = blockIdx.x;
    double s = 0.0;
    for (int b = threadIdx.x; b < r.blocks; b += 256) s += r.partial[(int64_t)b * nf + f];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    s = red[0];
    if (f < r.A) {
        r.grad_log_std[f] = (float)(s - (double)r.entropy_coef);
    } else {
        const int k = f - r.A;
        const double mean = s / (double)r.Mb;
        r.mb_stats[k] = mean;
    }
}

__global__ __launch_bounds__(256) void finalize_kernel(FinalizeArgs f)
{
    __shared__ double red[256];
    double s = 0.0;
    for (int b = threadIdx.x; b < f.norm_blocks; b += 256) s += f.norm_partial[b];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    const double norm = sqrt(red[0]);
    double scale = 1.0;
    if (f.max_grad_norm > 0.0f) {
        const double coef = (double)f.max_grad_norm / (norm + 1e-6);
        if (coef < 1.0) scale = coef;
    }
    const double kl = f.mb_stats[2];
    float lr = *f.lr;
    if (f.desired_kl > 0.0f) {
        if (kl > 2.0 * f.desired_kl) lr = fmaxf(f.lr_min, lr / 1.5f);
        else if (kl > 0.0 && kl < 0.5 * f.desired_kl) lr = fminf(f.lr_max, lr * 1.5f);
    }
    *f.lr = lr;
    const int step = *f.step + 1;
    *f.step = step;
    f.opt->scale = (float)scale;
    f.opt->lr = lr;
    f.opt->bc1 = (float)(1.0 - pow((double)f.beta1, (double)step));
    f.opt->bc2 = (float)(1.0 - pow((double)f.beta2, (double)step));
    if (f.stats) {
        f.stats[IM_PPO_LOSS_PI] += f.mb_stats[0];
        f.stats[IM_PPO_LOSS_V] += f.mb_stats[1];
        f.stats[IM_PPO_KL] += f.mb_stats[2];
        f.stats[IM_PPO_CLIP_FRAC] += f.mb_stats[3];
        f.stats[IM_PPO_GRAD_NORM] += norm;
        f.stats[IM_PPO_MINIBATCHES] += 1.0;
        f.stats[IM_PPO_LR] = (double)lr;
    }
}

__global__ __launch_bounds__(256) void adam_kernel(float *__restrict__ x, float *__restrict__ m,
                                                   float *__restrict__ v,
                                                   const float *__restrict__ g, int64_t P,
                                                   const OptScalars *__restrict__ o, float beta1,
                                                   float beta2, float eps)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= P) return;
    const float gi = g[i] * o->scale;
    const float mi = beta1 * m[i] + (1.0f - beta1) * gi;
    const float vi = beta2 * v[i] + (1.0f - beta2) * gi * gi;
    m[i] = mi;
    v[i] = vi;
    x[i] -= o->lr * (mi / o->bc1) / (sqrtf(vi / o->bc2) + eps);
}

// ---------------------------------------------------------------------------
// Weight refresh from the float32 masters: the training copies W [Mp][Kp]
// and W^T [Kp][Mp] (bf16), and the rollout's packed copy [M_pad][K_pad]
// (roll_bf16 1: bf16; 2: float32 holding the bf16-rounded value; 0:
// float32) with its bias; padding stays zero.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void repack_kernel(RepackArgs r)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)r.out * r.in) return;
    const int o = (int)(idx / r.in), i = (int)(idx % r.in);
    const float w = r.W[idx];
    const uint16_t h = f32_to_bf16_rne(w);
    if (r.wt) r.wt[(int64_t)o * r.Kp + i] = h;
    if (r.wtt) r.wtt[(int64_t)i * r.Mp + o] = h;
    if (r.roll) {
        if (r.roll_bf16 == 1) ((uint16_t *)r.roll)[(int64_t)o * r.roll_K + i] = h;
        else if (r.roll_bf16 == 2) ((float *)r.roll)[(int64_t)o * r.roll_K + i] = bf16_to_f32(h);
        else ((float *)r.roll)[(int64_t)o * r.roll_K + i] = w;
    }
    if (r.rollf) r.rollf[frag_index(o, i, r.roll_K / 64)] = h;
    if (i == 0) {
        if (r.bias_train) r.bias_train[o] = r.b[o];
        if (r.bias_roll) r.bias_roll[o] = r.b[o];
    }
}

// ---------------------------------------------------------------------------
// Host-side launchers.
// ---------------------------------------------------------------------------
hipError_t launch_tgemm(bool bt, int epi, const TGemm &g, int splits, hipStream_t s)
{
    // 256-row tiles of 8 waves and 256-column tiles where the shape allows
    const bool bigm = g.M % 256 == 0, bign = tgemm_bn(g.N) == 256;
    const int bm = bigm ? 256 : 128, bn = bign ? 256 : 128;
    const dim3 grid((unsigned)((g.M / bm) * (g.N / bn)), (unsigned)splits);
#define IM_TG(B, E)                                                                            \
    do {                                                                                      \
        if (bigm && bign) hipLaunchKernelGGL((tgemm_kernel<B, E, 4, 256>), grid, dim3(512), 0, s, g); \
        else if (bigm) hipLaunchKernelGGL((tgemm_kernel<B, E, 4, 128>), grid, dim3(512), 0, s, g);    \
        else if (bign) hipLaunchKernelGGL((tgemm_kernel<B, E, 2, 256>), grid, dim3(256), 0, s, g);    \
        else hipLaunchKernelGGL((tgemm_kernel<B, E, 2, 128>), grid, dim3(256), 0, s, g);              \
    } while (0)
    if (bt) {
        if (epi == T_HIDDEN) IM_TG(true, T_HIDDEN);
        else if (epi == T_MASK) IM_TG(true, T_MASK);
        else if (epi == T_LINEAR) IM_TG(true, T_LINEAR);
        else return hipErrorInvalidValue;
    } else {
        if (epi == T_PARTIAL) IM_TG(false, T_PARTIAL);
        else return hipErrorInvalidValue;
    }
#undef IM_TG
    return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(gather_kernel, dim3((unsigned)((a.chunks_pad + 3) / 4)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_head_forward(const uint16_t *h, int K, int64_t Mb, const float *w, const float *b,
                               float *v, hipStream_t s)
{
    hipLaunchKernelGGL(head_forward_kernel, dim3((unsigned)((Mb / 8 + 255) / 256)), dim3(256), 0, s, h, K,
                       Mb, w, b, v);
    return hipGetLastError();
}

hipError_t launch_head_backward(const uint16_t *h, int K, int rows, int64_t Mb, const float *w,
                                const float *dv, uint16_t *dz, double *pw, double *pb, hipStream_t s)
{
    // Mb is a multiple of 256: 8 samples per thread
    hipLaunchKernelGGL(head_backward_kernel, dim3((unsigned)((Mb / 8 + 255) / 256), (unsigned)rows),
                       dim3(256), 0, s, h, K, Mb, w, dv, dz, pw, pb);
    return hipGetLastError();
}

hipError_t launch_rowsum(bool bf16, const void *x, int rows, int64_t Mb, const float *y, double *part,
                         float *out, hipStream_t s)
{
    if (rows <= 0) return hipSuccess;
    // about 2048 blocks; segments of at least 2048 samples
    int parts = (2048 + rows - 1) / rows;
    while (parts > 1 && (Mb % ((int64_t)parts * 256) != 0 || Mb / parts < 2048)) --parts;
    const dim3 grid((unsigned)rows, (unsigned)parts);
    if (bf16)
        hipLaunchKernelGGL(rowsum_kernel<true>, grid, dim3(256), 0, s, x, Mb, y, parts, part);
    else
        hipLaunchKernelGGL(rowsum_kernel<false>, grid, dim3(256), 0, s, x, Mb, y, parts, part);
    hipLaunchKernelGGL(rowsum_finish_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, part,
                       rows, parts, out);
    return hipGetLastError();
}

hipError_t launch_rowsum_finish(const double *part, int rows, int parts, float *out, hipStream_t s)
{
    if (rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(rowsum_finish_rows_kernel, dim3((unsigned)rows), dim3(256), 0, s, part, parts, out);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float *P, int S, int64_t M, int64_t N, int rows, int cols,
                                float *out, hipStream_t s)
{
    const int64_t n = (int64_t)rows * cols;
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, P, S, M,
                       N, rows, cols, out);
    return hipGetLastError();
}

hipError_t launch_loss(const LossArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(loss_kernel, dim3((unsigned)(a.Mb_pad / 256)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_loss_reduce(const LossReduceArgs &r, hipStream_t s)
{
    hipLaunchKernelGGL(loss_reduce_kernel, dim3((unsigned)(r.A + LOSS_STATS)), dim3(256), 0, s, r);
    return hipGetLastError();
}

hipError_t launch_optimizer(const float *grad, int64_t P, double *norm_partial, int norm_blocks,
                            const FinalizeArgs &f, float *x, float *m, float *v, hipStream_t s)
{
    hipLaunchKernelGGL(norm_kernel, dim3((unsigned)norm_blocks), dim3(256), 0, s, grad, P, norm_partial);
    hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(256), 0, s, f);
    hipLaunchKernelGGL(adam_kernel, dim3((unsigned)((P + 255) / 256)), dim3(256), 0, s, x, m, v, grad, P,
                       f.opt, f.beta1, f.beta2, f.eps);
    return hipGetLastError();
}

hipError_t launch_norm(const float *grad, int64_t P, double *norm_partial, int norm_blocks,
                       hipStream_t s)
{
    hipLaunchKernelGGL(norm_kernel, dim3((unsigned)norm_blocks), dim3(256), 0, s, grad, P, norm_partial);
    return hipGetLastError();
}

hipError_t launch_repack(const RepackArgs &r, hipStream_t s)
{
    const int64_t n = (int64_t)r.out * r.in;
    hipLaunchKernelGGL(repack_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, r);
    return hipGetLastError();
}

}  // namespace im
