// device_math.h -- fp32 vector/quaternion algebra, counter-based random
// numbers and small polynomial kernels used by the env and policy kernels.
// Quaternions are (w, x, y, z), Hamilton product, active rotations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace im {

struct f3 {
    float x, y, z;
};
struct q4 {
    float w, x, y, z;
};

__device__ __forceinline__ f3 mk3(float x, float y, float z) { return f3{x, y, z}; }
__device__ __forceinline__ f3 operator+(f3 a, f3 b) { return f3{a.x + b.x, a.y + b.y, a.z + b.z}; }
__device__ __forceinline__ f3 operator-(f3 a, f3 b) { return f3{a.x - b.x, a.y - b.y, a.z - b.z}; }
__device__ __forceinline__ f3 operator*(float s, f3 a) { return f3{s * a.x, s * a.y, s * a.z}; }
__device__ __forceinline__ float dot3(f3 a, f3 b) { return a.x * b.x + a.y * b.y + a.z * b.z; }
__device__ __forceinline__ f3 cross3(f3 a, f3 b)
{
    return f3{a.y * b.z - a.z * b.y, a.z * b.x - a.x * b.z, a.x * b.y - a.y * b.x};
}

__device__ __forceinline__ q4 qmul(q4 a, q4 b)
{
    return q4{a.w * b.w - a.x * b.x - a.y * b.y - a.z * b.z,
              a.w * b.x + a.x * b.w + a.y * b.z - a.z * b.y,
              a.w * b.y - a.x * b.z + a.y * b.w + a.z * b.x,
              a.w * b.z + a.x * b.y - a.y * b.x + a.z * b.w};
}

// R(q) v for a unit q: v + w t + u x t with t = 2 u x v.
__device__ __forceinline__ q4 qconj(q4 a) { return q4{a.w, -a.x, -a.y, -a.z}; }
// rotation angle in [0, pi] of a unit quaternion (either sign)
__device__ __forceinline__ float qangle(q4 q)
{
    return 2.0f * atan2f(sqrtf(q.x * q.x + q.y * q.y + q.z * q.z), fabsf(q.w));
}
__device__ __forceinline__ f3 qrot(q4 q, f3 v)
{
    f3 u{q.x, q.y, q.z};
    f3 t = 2.0f * cross3(u, v);
    return v + q.w * t + cross3(u, t);
}

// sin and cos on [0, pi/2] from their Taylor series (truncation error below
// 1e-9 there), evaluated with Horner's rule.  Slerp only needs angles in
// this range: after the hemisphere flip the angle between two unit
// quaternions is at most pi/2 and the blend weight is in [0, 1].
__device__ __forceinline__ void sincos_q1(float x, float *s, float *c)
{
    const float x2 = x * x;
    float ps = 1.0f / 6227020800.0f;          // 1/13!
    ps = ps * x2 - 1.0f / 39916800.0f;        // 1/11!
    ps = ps * x2 + 1.0f / 362880.0f;          // 1/9!
    ps = ps * x2 - 1.0f / 5040.0f;            // 1/7!
    ps = ps * x2 + 1.0f / 120.0f;             // 1/5!
    ps = ps * x2 - 1.0f / 6.0f;               // 1/3!
    *s = x + (x * x2) * ps;
    float pc = -1.0f / 87178291200.0f;        // 1/14!
    pc = pc * x2 + 1.0f / 479001600.0f;       // 1/12!
    pc = pc * x2 - 1.0f / 3628800.0f;         // 1/10!
    pc = pc * x2 + 1.0f / 40320.0f;           // 1/8!
    pc = pc * x2 - 1.0f / 720.0f;             // 1/6!
    pc = pc * x2 + 1.0f / 24.0f;              // 1/4!
    pc = pc * x2 - 0.5f;                      // 1/2!
    *c = 1.0f + x2 * pc;
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of the
// two-multiplier round function, Weyl-sequence key schedule.  Each round's
// products are formed as full 64-bit products (one v_mad_u64_u32 each
// instead of separate low and high multiplies).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint4 philox4x32_10(uint4 ctr, uint32_t k0, uint32_t k1)
{
    uint32_t c0 = ctr.x, c1 = ctr.y, c2 = ctr.z, c3 = ctr.w;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        c0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        c1 = (uint32_t)p1;
        c2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        c3 = (uint32_t)p0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return make_uint4(c0, c1, c2, c3);
}

// Word -> (0, 1): odd multiples of 2^-24 (exact in fp32).
__device__ __forceinline__ float uniform_open(uint32_t x)
{
    return (float)(2u * (x >> 9) + 1u) * 0x1p-24f;
}

// Box-Muller: two words -> two standard normals (cos, sin branch).  The
// hardware sine and cosine take the angle in revolutions, so sin(2 pi v) is
// one instruction on v itself (measured max abs error 1.3e-7 over the open
// grid of v); the square root is the hardware one (1.5 ulp); the logarithm
// stays the accurate library one (ln u near u = 1 is a small difference).
__device__ __forceinline__ void box_muller(uint32_t a, uint32_t b, float *z0, float *z1)
{
    const float u = uniform_open(a), v = uniform_open(b);
    const float r = __builtin_amdgcn_sqrtf(-2.0f * logf(u));
    *z0 = r * __builtin_amdgcn_cosf(v);
    *z1 = r * __builtin_amdgcn_sinf(v);
}

__device__ __forceinline__ void normals4(uint64_t seed, uint32_t e, uint32_t n, uint32_t blk,
                                         uint32_t tag, float z[4])
{
    const uint4 x = philox4x32_10(make_uint4(e, n, blk, tag), (uint32_t)seed,
                                  (uint32_t)(seed >> 32));
    box_muller(x.x, x.y, &z[0], &z[1]);
    box_muller(x.z, x.w, &z[2], &z[3]);
}

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Two fp32 values -> packed bf16 pair (a in the low half), rounded to nearest
// even by the hardware conversion (v_cvt_pk_bf16_f32); equal to two
// f32_to_bf16_rne for finite inputs, a quiet NaN for NaN.
typedef __bf16 im_bf16x2_t __attribute__((ext_vector_type(2)));
typedef float im_f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b)
{
    const im_f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, im_bf16x2_t));
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

}  // namespace im
