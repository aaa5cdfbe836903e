// env_kernels.hip -- the fused environment step and its companions on gfx950.
//
// One thread per environment.  Every per-env array is structure-of-arrays
// with the env index fastest, so each load and store of a wavefront touches
// 64 consecutive floats (256 contiguous bytes).  The skeleton table is read
// with wave-uniform loads; reference segments are gathered from a
// cache-resident table (one contiguous record per segment, read
// sequentially in preorder).
//
// Forward kinematics walks the bodies in depth-first preorder: a body's
// parent is the previous body, or a branch point whose frame was parked in
// LDS.  For small batches the fused step runs every env on several threads
// (the same lane of consecutive wavefronts), each walking the bodies of one
// part of the skeleton plus their ancestors (two halves, or one root-to-leaf
// path each); the partial error sums are combined through LDS.
//
// Reference positions are kept relative to an anchor (the clip root
// position at frame i0) and the simulator positions are differenced against
// the same anchor, so the reward's position errors are formed from numbers
// of body-size magnitude even when the character has travelled far from the
// origin.
#include <hip/hip_runtime.h>

#include "device_math.h"
#include "launch.h"

namespace im {

struct Frame {
    q4 Q;  // world orientation
    f3 P;  // position relative to the segment anchor
    f3 W;  // world angular velocity
    f3 V;  // world linear velocity
};

// Frames of branch points (bodies with two or more children) are parked in
// LDS, laid out [slot][component][thread] so that every access of a
// wavefront is conflict-free.  In preorder a body's parent is the previous
// body except right after a leaf, when it is a branch point: LDS is touched
// only at those few events.
template <int NC>
struct LdsStack {
    float *base;  // this thread's column
    int bs;       // threads per block
    __device__ __forceinline__ void put(int slot, const float (&v)[NC]) const
    {
        float *p = base + slot * NC * bs;
#pragma unroll
        for (int c = 0; c < NC; ++c) p[c * bs] = v[c];
    }
    __device__ __forceinline__ void get(int slot, float (&v)[NC]) const
    {
        const float *p = base + slot * NC * bs;
#pragma unroll
        for (int c = 0; c < NC; ++c) v[c] = p[c * bs];
    }
};

extern __shared__ float im_lds[];

__device__ __forceinline__ void pack_frame(const Frame &f, float (&v)[13])
{
    v[0] = f.Q.w; v[1] = f.Q.x; v[2] = f.Q.y; v[3] = f.Q.z;
    v[4] = f.P.x; v[5] = f.P.y; v[6] = f.P.z;
    v[7] = f.W.x; v[8] = f.W.y; v[9] = f.W.z;
    v[10] = f.V.x; v[11] = f.V.y; v[12] = f.V.z;
}
__device__ __forceinline__ Frame unpack_frame(const float (&v)[13])
{
    Frame f;
    f.Q = q4{v[0], v[1], v[2], v[3]};
    f.P = mk3(v[4], v[5], v[6]);
    f.W = mk3(v[7], v[8], v[9]);
    f.V = mk3(v[10], v[11], v[12]);
    return f;
}

__device__ __forceinline__ q4 slerp_basis(float4 a, float4 u, float theta)
{
    float s, c;
    sincos_q1(theta, &s, &c);
    return q4{c * a.x + s * u.x, c * a.y + s * u.y, c * a.z + s * u.z, c * a.w + s * u.w};
}

// Root of the reference at blend alpha of a segment record.
__device__ __forceinline__ Frame root_frame(const float4 *rec, float alpha, f3 *anchor)
{
    const float4 r0 = rec[0], r1 = rec[1], r2 = rec[2], ra = rec[3], ru = rec[4], r5 = rec[5];
    *anchor = mk3(r0.x, r0.y, r0.z);
    Frame f;
    f.P = alpha * mk3(r0.w, r1.x, r1.y);
    f.V = mk3(r1.z, r1.w, r2.x);
    f.W = mk3(r2.y, r2.z, r2.w);
    f.Q = slerp_basis(ra, ru, alpha * r5.x);
    return f;
}

// Child frame: Q = Qp q, P = Pp + R(Qp) off, W = Wp + R(Qp) w, V = Vp + Wp x (P - Pp).
__device__ __forceinline__ Frame child_frame(const Frame &p, const float4 *rec, float alpha,
                                             f3 off, int jt)
{
    Frame f;
    const f3 r = qrot(p.Q, off);
    f.P = p.P + r;
    f.V = p.V + cross3(p.W, r);
    if (jt == IM_JOINT_FIXED) {
        f.Q = p.Q;
        f.W = p.W;
    } else {
        const float4 a = rec[0], u = rec[1], w = rec[2];
        f.Q = qmul(p.Q, slerp_basis(a, u, alpha * w.w));
        f.W = p.W + qrot(p.Q, mk3(w.x, w.y, w.z));
    }
    return f;
}

// Forward kinematics of one reference segment record in preorder, over a walk
// table T (the whole skeleton, or one part of it): visit(i, body, own, frame,
// anchor, data, q_joint, w_joint) is called for every position i (q_joint, w_joint:
// the reference joint rotation and joint angular velocity in the parent frame;
// the root's world values).  A ring of R slots keeps the segment record and
// the per-body data returned by load(body) of the next R - 1 positions in
// flight while one position is processed: position i takes slot (i - 1) % R,
// which is then refilled with position i + R.  The loop is unrolled by R so
// that each slot stays in fixed registers; a rotating buffer (next -> current)
// would copy registers whose loads are still in flight, and each copy waits
// for them, which costs a whole memory latency per position.  Positions past
// the end refetch the walk's last body, so that every load is unconditional
// and inside the tables.
struct NoData {
};

using PartWalk = SkelTab::PartWalk;

// The walk tables: the whole skeleton (position p's segment record is p) or
// one part walk (its record is rec[p]); both have body, pslot, bslot, jtype
// and offset per position.  The walk reads them through the constant address
// space: they are written only when a context is created, and so their reads
// stay scalar loads (counted apart from the vector memory operations) also
// where the walk itself stores (reset walks); read as ordinary global memory
// next to those stores they became vector loads, each waiting for every
// store and load issued before it.
#define IM_CONST_AS __attribute__((address_space(4)))
__device__ __forceinline__ int walk_len(const IM_CONST_AS SkelTab *t) { return t->B; }
__device__ __forceinline__ int walk_len(const IM_CONST_AS PartWalk *t) { return t->n; }
__device__ __forceinline__ int walk_rec(const IM_CONST_AS SkelTab *, int p) { return p; }
__device__ __forceinline__ int walk_rec(const IM_CONST_AS PartWalk *t, int p) { return t->rec[p]; }
__device__ __forceinline__ bool walk_own(const IM_CONST_AS SkelTab *, int) { return true; }
__device__ __forceinline__ bool walk_own(const IM_CONST_AS PartWalk *t, int p) { return t->own[p] != 0; }

template <int R, class D, class T, class Load, class Visit>
__device__ __forceinline__ void walk_ring(const T *tg, const float4 *rec, float alpha, Load &&load,
                                          Visit &&visit)
{
    const IM_CONST_AS T *t = (const IM_CONST_AS T *)tg;
    const LdsStack<13> st{im_lds + threadIdx.x, (int)blockDim.x};
    float buf[13];
    const int n = walk_len(t);
    const float4 *jr = rec + 6;
    struct Slot {
        D d;
        float4 a, u, w;
    };
    auto fetch = [&](int p, Slot &s) {
        const int q = p < n ? p : n - 1;
        s.d = load(t->body[q]);
        const float4 *r = jr + 3 * (walk_rec(t, q) - 1);
        s.a = r[0];
        s.u = r[1];
        s.w = r[2];
    };
    const D d0 = load(0);
    Slot sl[R];
#pragma unroll
    for (int j = 0; j < R; ++j) fetch(1 + j, sl[j]);
    f3 A;
    Frame cur = root_frame(rec, alpha, &A);
    visit(0, t->body[0], walk_own(t, 0), cur, A, d0, cur.Q, cur.W);
    if (t->bslot[0] >= 0) {
        pack_frame(cur, buf);
        st.put(t->bslot[0], buf);
    }
    auto step = [&](int i, const Slot &s) {
        if (t->pslot[i] >= 0) {
            st.get(t->pslot[i], buf);
            cur = unpack_frame(buf);
        }
        const f3 off = mk3(t->offset[i][0], t->offset[i][1], t->offset[i][2]);
        // child frame from the prefetched record (same arithmetic as child_frame)
        Frame c;
        const f3 r = qrot(cur.Q, off);
        c.P = cur.P + r;
        c.V = cur.V + cross3(cur.W, r);
        q4 ql = q4{1.0f, 0.0f, 0.0f, 0.0f};
        f3 wl = mk3(0.0f, 0.0f, 0.0f);
        if (t->jtype[i] == IM_JOINT_FIXED) {
            c.Q = cur.Q;
            c.W = cur.W;
        } else {
            ql = slerp_basis(s.a, s.u, alpha * s.w.w);
            wl = mk3(s.w.x, s.w.y, s.w.z);
            c.Q = qmul(cur.Q, ql);
            c.W = cur.W + qrot(cur.Q, wl);
        }
        cur = c;
        visit(i, t->body[i], walk_own(t, i), cur, A, s.d, ql, wl);
        if (t->bslot[i] >= 0) {
            pack_frame(cur, buf);
            st.put(t->bslot[i], buf);
        }
    };
    int i = 1;
    for (; i + R <= n; i += R) {
#pragma unroll
        for (int j = 0; j < R; ++j) {
            step(i + j, sl[j]);
            fetch(i + j + R, sl[j]);
        }
    }
#pragma unroll
    for (int j = 0; j < R - 1; ++j)
        if (i + j < n) step(i + j, sl[j]);
}

constexpr int WALK_RING = 3;

// visit(i, body, frame, anchor, data, q_joint, w_joint) for every preorder
// position i of the skeleton.
template <class D, class Load, class Visit>
__device__ __forceinline__ void walk_prefetch(const SkelTab *__restrict__ sk, const float4 *rec,
                                              float alpha, Load &&load, Visit &&visit)
{
    walk_ring<WALK_RING, D>(sk, rec, alpha, load,
                            [&](int i, int b, bool, const Frame &f, f3 A, const D &d, q4 ql, f3 wl) {
                                visit(i, b, f, A, d, ql, wl);
                            });
}

// Discrete phase -> (i0, alpha), fp32 without contraction.  phi_ev is
// clamped to [0, 1] (a NaN phase maps to 0) so that a corrupt env state can
// never index outside the segment table; valid phases are unchanged.
__device__ __forceinline__ void phase_index(float phi_ev, const ClipTab &ci, int *i0, float *alpha)
{
#pragma clang fp contract(off)
    phi_ev = phi_ev > 0.0f ? (phi_ev < 1.0f ? phi_ev : 1.0f) : 0.0f;
    const float s = phi_ev * ci.fm1;
    int i = (int)s;
    i = i < ci.F - 2 ? i : ci.F - 2;
    *i0 = i;
    *alpha = s - (float)i;
}

// Clip index of an env, clamped into the table for memory safety.
__device__ __forceinline__ int safe_clip(int k, int n_clips)
{
    return k < 0 ? 0 : (k >= n_clips ? n_clips - 1 : k);
}

struct Heading {
    float c, s, ox, oy;
};

__device__ __forceinline__ Heading heading_of(q4 q, f3 p)
{
    // forward axis R(q) x projected on the ground plane
    const float fx = 1.0f - 2.0f * (q.y * q.y + q.z * q.z);
    const float fy = 2.0f * (q.x * q.y + q.w * q.z);
    const float h2 = fx * fx + fy * fy;
    Heading h;
    if (h2 < 1e-12f) {
        h.c = 1.0f;
        h.s = 0.0f;
    } else {
        const float inv = rsqrtf(h2);
        h.c = fx * inv;
        h.s = fy * inv;
    }
    h.ox = p.x;
    h.oy = p.y;
    return h;
}

__device__ __forceinline__ f3 ld3(const float *a, int b, int64_t ld, int64_t e)
{
    const float *p = a + (int64_t)(3 * b) * ld + e;
    return mk3(p[0], p[ld], p[2 * ld]);
}
__device__ __forceinline__ q4 ld4(const float *a, int b, int64_t ld, int64_t e)
{
    const float *p = a + (int64_t)(4 * b) * ld + e;
    return q4{p[0], p[ld], p[2 * ld], p[3 * ld]};
}
__device__ __forceinline__ void st3(float *a, int b, int64_t ld, int64_t e, f3 v)
{
    float *p = a + (int64_t)(3 * b) * ld + e;
    p[0] = v.x;
    p[ld] = v.y;
    p[2 * ld] = v.z;
}
__device__ __forceinline__ void st4(float *a, int b, int64_t ld, int64_t e, q4 q)
{
    float *p = a + (int64_t)(4 * b) * ld + e;
    p[0] = q.w;
    p[ld] = q.x;
    p[2 * ld] = q.y;
    p[3 * ld] = q.z;
}

// 9 observation rows of a frame in the heading frame, starting at row `row`:
// position, then the first two columns of the rotation matrix.
__device__ __forceinline__ void write_frame9(float *obs, int64_t ld, int64_t e, int row,
                                             const Heading &h, f3 P, q4 Q)
{
    float *o = obs + (int64_t)row * ld + e;
    const float px = P.x - h.ox, py = P.y - h.oy;
    o[0] = h.c * px + h.s * py;
    o[ld] = h.c * py - h.s * px;
    o[2 * ld] = P.z;
    const float c0x = 1.0f - 2.0f * (Q.y * Q.y + Q.z * Q.z);
    const float c0y = 2.0f * (Q.x * Q.y + Q.w * Q.z);
    const float c0z = 2.0f * (Q.x * Q.z - Q.w * Q.y);
    const float c1x = 2.0f * (Q.x * Q.y - Q.w * Q.z);
    const float c1y = 1.0f - 2.0f * (Q.x * Q.x + Q.z * Q.z);
    const float c1z = 2.0f * (Q.y * Q.z + Q.w * Q.x);
    o[3 * ld] = h.c * c0x + h.s * c0y;
    o[4 * ld] = h.c * c0y - h.s * c0x;
    o[5 * ld] = c0z;
    o[6 * ld] = h.c * c1x + h.s * c1y;
    o[7 * ld] = h.c * c1y - h.s * c1x;
    o[8 * ld] = c1z;
}

// The 15 observation rows of a body in the heading frame: position, the first
// two columns of the rotation matrix, linear and angular velocity.
__device__ __forceinline__ void obs_body_rows(const Heading &h, f3 P, q4 Q, f3 V, f3 W,
                                              float (&o)[15])
{
    const float px = P.x - h.ox, py = P.y - h.oy;
    o[0] = h.c * px + h.s * py;
    o[1] = h.c * py - h.s * px;
    o[2] = P.z;
    const float c0x = 1.0f - 2.0f * (Q.y * Q.y + Q.z * Q.z);
    const float c0y = 2.0f * (Q.x * Q.y + Q.w * Q.z);
    const float c0z = 2.0f * (Q.x * Q.z - Q.w * Q.y);
    const float c1x = 2.0f * (Q.x * Q.y - Q.w * Q.z);
    const float c1y = 1.0f - 2.0f * (Q.x * Q.x + Q.z * Q.z);
    const float c1z = 2.0f * (Q.y * Q.z + Q.w * Q.x);
    o[3] = h.c * c0x + h.s * c0y;
    o[4] = h.c * c0y - h.s * c0x;
    o[5] = c0z;
    o[6] = h.c * c1x + h.s * c1y;
    o[7] = h.c * c1y - h.s * c1x;
    o[8] = c1z;
    o[9] = h.c * V.x + h.s * V.y;
    o[10] = h.c * V.y - h.s * V.x;
    o[11] = V.z;
    o[12] = h.c * W.x + h.s * W.y;
    o[13] = h.c * W.y - h.s * W.x;
    o[14] = W.z;
}

__device__ __forceinline__ void store_obs_body(float *obs, int64_t ld, int64_t e, int b,
                                               const float (&o)[15])
{
    float *p = obs + (int64_t)(15 * b) * ld + e;
#pragma unroll
    for (int r = 0; r < 15; ++r) p[r * ld] = o[r];
}

// 15 observation rows of body b in the heading frame.
__device__ __forceinline__ void write_obs_body(float *obs, int64_t ld, int64_t e, int b,
                                               const Heading &h, f3 P, q4 Q, f3 V, f3 W)
{
    float o[15];
    obs_body_rows(h, P, Q, V, W, o);
    store_obs_body(obs, ld, e, b, o);
}

struct SimFull {
    f3 P;
    q4 Q;
    f3 V, W;
};

// Observation of env e from its (post-reset) sim state.  A ring of three
// slots holds the sim state of the next bodies: body b's rows are formed from
// its slot, the slot is refilled with body b + 3, and only then are the rows
// stored.  A wave counts its loads and stores in one in-order queue, so the
// loads of a body issued after the previous body's stores (the plain loop)
// wait for those stores to complete; issued before them, they wait only for
// the stores of three bodies back.  Bodies past the last refetch it.
__device__ __forceinline__ void obs_from_sim(const EnvArgs &a, int64_t e, float phase)
{
    const int64_t ld = a.ld;
    const int B = a.sk->B;
    auto fetch = [&](int b, SimFull &sf) {
        const int q = b < B ? b : B - 1;
        sf.P = ld3(a.pos, q, ld, e);
        sf.Q = ld4(a.quat, q, ld, e);
        sf.V = ld3(a.linvel, q, ld, e);
        sf.W = ld3(a.angvel, q, ld, e);
    };
    SimFull sl[3];
#pragma unroll
    for (int j = 0; j < 3; ++j) fetch(j, sl[j]);
    const Heading h = heading_of(sl[0].Q, sl[0].P);
    int b = 0;
    for (; b + 3 <= B; b += 3) {
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            float o[15];
            obs_body_rows(h, sl[j].P, sl[j].Q, sl[j].V, sl[j].W, o);
            // the refill stays after the rows are formed, so that the slot
            // keeps its registers across the loop
            __builtin_amdgcn_sched_barrier(0);
            fetch(b + j + 3, sl[j]);
            __builtin_amdgcn_sched_barrier(0);
            store_obs_body(a.obs, ld, e, b + j, o);
        }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
        if (b + j < B) write_obs_body(a.obs, ld, e, b + j, h, sl[j].P, sl[j].Q, sl[j].V, sl[j].W);
    a.obs[(int64_t)(15 * B) * ld + e] = phase;
}

// Observation rows after the phase: the reference frames of the root and the
// end effectors at the next obs_future control steps of clip k (phase_j =
// phase_{j-1} + dphi in fp32, evaluated at min(phase_j, 1)), in the heading
// frame h of the env's current (post-reset) sim root, then the previous action
// (zero for an env reset in this call).  This call writes future frames
// j = j0, j0 + js, ... (j counted from 0) and, with prev, the action rows.
__device__ __forceinline__ void obs_extras(const EnvArgs &a, int64_t e, int k, float ph,
                                           bool reset, const Heading &h, int j0, int js, bool prev)
{
    const int64_t ld = a.ld;
    const SkelTab *__restrict__ sk = a.sk;
    const IM_CONST_AS SkelTab *skc = (const IM_CONST_AS SkelTab *)sk;  // scalar reads next to stores
    const int rows_f = 9 * (1 + skc->n_ee);
    const ClipTab ci = a.clips[k];
    float phj = ph;
    for (int j = 0; j < a.obs_future; ++j) {
        {
#pragma clang fp contract(off)
            phj = phj + ci.dphi;
        }
        if (j < j0 || (j - j0) % js != 0) continue;
        int i0;
        float al;
        phase_index(phj < 1.0f ? phj : 1.0f, ci, &i0, &al);
        const float4 *rec = a.seg + ci.seg_base + (int64_t)i0 * seg_stride(sk->B);
        const int base = a.obs_base + j * rows_f;
        walk_prefetch<NoData>(sk, rec, al, [](int) { return NoData{}; },
                              [&](int i, int, const Frame &f, f3 A, const NoData &, q4, f3) {
            const int slot = skc->ee_slot[i];
            if (slot >= 0) write_frame9(a.obs, ld, e, base + 9 * slot, h, A + f.P, f.Q);
        });
    }
    if (prev) {
        const int row = a.obs_base + a.obs_future * rows_f;
        for (int c = 0; c < a.A; ++c)
            a.obs[(int64_t)(row + c) * ld + e] = reset ? 0.0f : a.prev_action[e * a.A + c];
    }
}

// The heading frame of env e's current sim root.
__device__ __forceinline__ Heading sim_heading(const EnvArgs &a, int64_t e)
{
    return heading_of(ld4(a.quat, 0, a.ld, e), ld3(a.pos, 0, a.ld, e));
}

// Reference state initialisation: the sim state of env e := the reference
// at (clip k, phase ph).
__device__ __forceinline__ void rsi(const EnvArgs &a, int64_t e, int k, float ph)
{
    const ClipTab ci = a.clips[k];
    int j0;
    float al;
    phase_index(ph, ci, &j0, &al);
    const float4 *rec = a.seg + ci.seg_base + (int64_t)j0 * seg_stride(a.sk->B);
    const int64_t ld = a.ld;
    walk_prefetch<NoData>(a.sk, rec, al, [](int) { return NoData{}; },
                          [&](int, int b, const Frame &f, f3 A, const NoData &, q4, f3) {
        st3(a.pos, b, ld, e, A + f.P);
        st4(a.quat, b, ld, e, f.Q);
        st3(a.linvel, b, ld, e, f.V);
        st3(a.angvel, b, ld, e, f.W);
    });
}

struct SimPV {
    f3 P, V;
};

// Forward kinematics over one part walk: visit(i, body, own, frame, anchor,
// data, joint rotation, joint angular velocity) for every position.  load(body)
// is called for every position, owned or not (an ancestor's data is what its
// owner's walk reads too, so it comes from the cache), so that the ring's
// loads stay unconditional; visit uses it for owned bodies only.
template <class D, class Load, class Visit>
__device__ __forceinline__ void walk_part(const PartWalk *__restrict__ w, const float4 *rec,
                                          float alpha, Load &&load, Visit &&visit)
{
    walk_ring<WALK_RING, D>(w, rec, alpha, load, visit);
}

// Observation rows of the bodies a part walk owns, from the sim state (env
// not reset); h = the heading of the sim root.  The same three-slot ring as
// obs_from_sim, over the walk's owned bodies.
__device__ __forceinline__ void obs_part_from_sim(const EnvArgs &a, const PartWalk *__restrict__ wg,
                                                  int64_t e, const Heading &h)
{
    const IM_CONST_AS PartWalk *w = (const IM_CONST_AS PartWalk *)wg;
    const int64_t ld = a.ld;
    const int n = w->n_own;
    if (n <= 0) return;
    auto fetch = [&](int j, SimFull &sf) {
        const int b = w->own_body[j < n ? j : n - 1];
        sf.P = ld3(a.pos, b, ld, e);
        sf.Q = ld4(a.quat, b, ld, e);
        sf.V = ld3(a.linvel, b, ld, e);
        sf.W = ld3(a.angvel, b, ld, e);
    };
    SimFull sl[3];
#pragma unroll
    for (int j = 0; j < 3; ++j) fetch(j, sl[j]);
    int i = 0;
    for (; i + 3 <= n; i += 3) {
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            float o[15];
            obs_body_rows(h, sl[j].P, sl[j].Q, sl[j].V, sl[j].W, o);
            __builtin_amdgcn_sched_barrier(0);
            fetch(i + j + 3, sl[j]);
            __builtin_amdgcn_sched_barrier(0);
            store_obs_body(a.obs, ld, e, w->own_body[i + j], o);
        }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
        if (i + j < n)
            write_obs_body(a.obs, ld, e, w->own_body[i + j], h, sl[j].P, sl[j].Q, sl[j].V, sl[j].W);
}

// Reference state initialisation of the bodies a part walk owns at (clip k,
// phase ph), and their observation rows from the same fp32 values the sim
// state receives (the heading from the root, which every walk visits first;
// it is returned).
__device__ __forceinline__ Heading rsi_obs_part(const EnvArgs &a, const PartWalk *__restrict__ w,
                                                int64_t e, int k, float ph)
{
    const ClipTab ci = a.clips[k];
    int j0;
    float al;
    phase_index(ph, ci, &j0, &al);
    const float4 *rec = a.seg + ci.seg_base + (int64_t)j0 * seg_stride(a.sk->B);
    const int64_t ld = a.ld;
    Heading h{};
    walk_part<NoData>(w, rec, al, [](int) { return NoData{}; },
                      [&](int i, int b, int own, const Frame &f, f3 A, const NoData &, q4, f3) {
        const f3 P = A + f.P;
        if (i == 0) h = heading_of(f.Q, P);
        if (!own) return;
        st3(a.pos, b, ld, e, P);
        st4(a.quat, b, ld, e, f.Q);
        st3(a.linvel, b, ld, e, f.V);
        st3(a.angvel, b, ld, e, f.W);
        write_obs_body(a.obs, ld, e, b, h, P, f.Q, f.V, f.W);
    });
    return h;
}

struct SimMul {
    f3 P, W, Wp;
    q4 Q, Qp;   // the body's and its parent's orientation
};

// Sim state of body b for the multiplicative reward: the joint rotations and
// joint angular velocities in the parent frame need the parent's orientation
// and angular velocity.
__device__ __forceinline__ SimMul load_mul(const EnvArgs &a, int b, int64_t e)
{
    const int64_t ld = a.ld;
    SimMul s;
    s.P = ld3(a.pos, b, ld, e);
    s.Q = ld4(a.quat, b, ld, e);
    s.W = ld3(a.angvel, b, ld, e);
    const int p = b > 0 ? a.sk->pbody[b] : 0;
    s.Qp = ld4(a.quat, p, ld, e);
    s.Wp = ld3(a.angvel, p, ld, e);
    return s;
}

// Error sums of the multiplicative reward.
struct MulErr {
    float jrot = 0.0f, jvel = 0.0f, eepos = 0.0f, eerot = 0.0f;
    f3 dc = mk3(0.0f, 0.0f, 0.0f);
    // body at walk position i, index b (b = 0: the root); qr, wr: its reference
    // joint rotation and joint angular velocity
    __device__ __forceinline__ void add(int b, bool leaf, float massw, const Frame &f, f3 A,
                                        const SimMul &sb, q4 qr, f3 wr)
    {
        q4 ql = sb.Q;
        f3 wl = sb.W;
        if (b > 0) {
            const q4 ip = qconj(sb.Qp);
            ql = qmul(ip, sb.Q);
            wl = qrot(ip, sb.W - sb.Wp);
        }
        const float th = qangle(qmul(qconj(qr), ql));
        jrot += th * th;
        const f3 dw = wl - wr;
        jvel += dot3(dw, dw);
        const f3 dp = (sb.P - A) - f.P;
        dc = dc + massw * dp;
        if (leaf) {
            eepos += dot3(dp, dp);
            const float te = qangle(qmul(qconj(f.Q), sb.Q));
            eerot += te * te;
        }
    }
    // the product of the five exponentials, as one
    __device__ __forceinline__ float reward(const EnvArgs &a) const
    {
        return expf(-(a.m_jrot * jrot + a.m_jvel * jvel + a.m_com * dot3(dc, dc) +
                      a.m_eepos * eepos + a.m_eerot * eerot));
    }
};

// The fused step for small batches: env e runs on P = a.n_parts threads, lane
// l of P consecutive wavefronts of its block, the p-th walking a.walks[p]
// (two halves of the skeleton, or its root-to-leaf paths).  The walk is
// wave-uniform, so its tables are read with scalar loads.  A block holds
// G = max(1, 4 / P) groups of 64 envs.  The partial error sums meet in LDS
// and every thread adds them in walk order, so all P threads hold the same
// bits.  More wavefronts than the one-thread kernel for the same envs, each
// with a shorter walk: below a few waves per SIMD that hides more of the
// walks' latency, above it the repeated ancestor work costs more.  Future
// reference frames of the observation are dealt round-robin to the walks.
// MUL: the multiplicative reward.
template <bool MUL>
__global__ __launch_bounds__(512) void env_step_parts_kernel(EnvArgs a)
{
    __shared__ float part[7][512];
    const int tid = threadIdx.x;
    const int P = a.n_parts;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int pw_i = wave % P, grp = wave / P;
    const int G = (int)(blockDim.x >> 6) / P;
    const int lane = tid & 63;
    const int64_t e = ((int64_t)blockIdx.x * G + grp) * 64 + lane;
    const bool active = e < a.n;      // the same for all P threads of an env
    const int64_t ld = a.ld;
    const SkelTab *__restrict__ sk = a.sk;
    const PartWalk *__restrict__ hw = &a.walks[pw_i];

    // 1. discrete state advance (fp32, exact contract), in every thread
    int k = 0, t1 = 0, i0 = 0;
    uint32_t n1 = 0;
    float phi1 = 0.0f, alpha = 0.0f;
    bool trunc = false;
    // 2.-3. reference FK and this walk's error sums against the sim state
    float e_pos = 0.0f, e_ee = 0.0f, e_vel = 0.0f;
    f3 dc = mk3(0.0f, 0.0f, 0.0f);
    MulErr me;
    // The root height is read before the barrier below: after it, the walk that
    // owns the root may already be writing a reset root state, and every thread
    // of the env must decide termination on the same (pre-reset) value.
    float z_root = 0.0f;
    if (active) {
        z_root = a.pos[2 * ld + e];
        k = safe_clip(a.env_clip[e], a.n_clips);
        const float phi = a.env_phase[e];
        t1 = a.env_t[e] + 1;
        n1 = a.env_n[e] + 1u;
        const ClipTab ci = a.clips[k];
        {
#pragma clang fp contract(off)
            phi1 = phi + ci.dphi;
        }
        trunc = phi1 >= 1.0f;
        phase_index(phi1 < 1.0f ? phi1 : 1.0f, ci, &i0, &alpha);
        const float4 *rec = a.seg + ci.seg_base + (int64_t)i0 * seg_stride(sk->B);
        if constexpr (!MUL) {
            auto load_pv = [&](int b) {
                SimPV s;
                s.P = ld3(a.pos, b, ld, e);
                s.V = ld3(a.linvel, b, ld, e);
                return s;
            };
            walk_part<SimPV>(hw, rec, alpha, load_pv,
                             [&](int i, int, int own, const Frame &f, f3 A, const SimPV &sb, q4,
                                 f3) {
                if (!own) return;
                const f3 dp = (sb.P - A) - f.P;
                const f3 dv = sb.V - f.V;
                const float x = dot3(dp, dp);
                e_pos += x;
                if (hw->leaf[i]) e_ee += x;
                dc = dc + hw->massw[i] * dp;
                e_vel += dot3(dv, dv);
            });
        } else {
            walk_part<SimMul>(hw, rec, alpha, [&](int b) { return load_mul(a, b, e); },
                              [&](int i, int b, int own, const Frame &f, f3 A, const SimMul &sb,
                                  q4 qr, f3 wr) {
                if (own) me.add(b, hw->leaf[i], hw->massw[i], f, A, sb, qr, wr);
            });
        }
    }
    // the walks' sums, added in walk order by every thread of the env
    const int nb = (int)blockDim.x;
    const int g0 = grp * P * 64 + lane;
    auto sum_parts = [&](int c) {
        float v = part[c][g0];
        for (int q = 1; q < P; ++q) v += part[c][g0 + q * 64];
        return v;
    };
    float r;
    if constexpr (!MUL) {
        part[0][tid] = e_pos;
        part[1][tid] = e_ee;
        part[2][tid] = e_vel;
        part[3][tid] = dc.x;
        part[4][tid] = dc.y;
        part[5][tid] = dc.z;
        __syncthreads();
        e_pos = sum_parts(0);
        e_ee = sum_parts(1);
        e_vel = sum_parts(2);
        dc = mk3(sum_parts(3), sum_parts(4), sum_parts(5));
        const float e_com = dot3(dc, dc);
        r = a.c_pose * expf(-(a.w_pos * e_pos + a.w_ee * e_ee)) +
            a.c_vel * expf(-(a.w_vel * e_vel)) + a.c_com * expf(-(a.w_com * e_com));
    } else {
        part[0][tid] = me.jrot;
        part[1][tid] = me.jvel;
        part[2][tid] = me.eepos;
        part[3][tid] = me.eerot;
        part[4][tid] = me.dc.x;
        part[5][tid] = me.dc.y;
        part[6][tid] = me.dc.z;
        __syncthreads();
        me.jrot = sum_parts(0);
        me.jvel = sum_parts(1);
        me.eepos = sum_parts(2);
        me.eerot = sum_parts(3);
        me.dc = mk3(sum_parts(4), sum_parts(5), sum_parts(6));
        r = me.reward(a);
    }
    (void)nb;
    if (!active) return;
    const bool term = (t1 > a.grace) && ((z_root < a.h_term) || !(r >= a.r_min));

    // 4. masked reset (the same draw in every thread of the env)
    int k_out = k, t_out = t1;
    float ph_out = phi1;
    const bool done = term || trunc;
    if (done) {
        const uint4 x = philox4x32_10(make_uint4((uint32_t)e, n1, 0u, 1u), (uint32_t)a.seed,
                                      (uint32_t)(a.seed >> 32));
        k_out = (int)(((uint64_t)x.x * (uint64_t)(uint32_t)a.n_clips) >> 32);
        ph_out = (float)(x.y >> 8) * 0x1p-24f;
        t_out = 0;
    }
    if (pw_i == 0) {
        a.env_clip[e] = k_out;
        a.env_phase[e] = ph_out;
        a.env_t[e] = t_out;
        a.env_n[e] = n1;
        a.reward[e] = r;
        a.term[e] = (uint8_t)term;
        a.trunc[e] = (uint8_t)trunc;
        if (a.ref_frame) a.ref_frame[e] = i0;
        a.obs[(int64_t)(15 * sk->B) * ld + e] = ph_out;
    }
    // 5. observation of the post-reset state: a reset env's rows come from the
    //    reference state written in the same walk, others from the sim state
    Heading h;
    if (done) {
        h = rsi_obs_part(a, hw, e, k_out, ph_out);
    } else {
        h = sim_heading(a, e);
        obs_part_from_sim(a, hw, e, h);
    }
    // future frames j = p, p + P, ...; the previous action in the last walk
    if (a.obs_future > 0 || a.obs_prev)
        obs_extras(a, e, k_out, ph_out, done, h, pw_i, P, a.obs_prev && pw_i == P - 1);
}

// The fused step, one thread per env (large batches and the training terms).
// MUL: the multiplicative reward.
template <bool MUL>
__global__ __launch_bounds__(256) void env_step_kernel(EnvArgs a)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool active = e < a.n;
    const int64_t ld = a.ld;
    const SkelTab *__restrict__ sk = a.sk;
    float ph_out = 0.0f;
    int k_fin = 0;
    bool reset = false;

    if (active) {
        // 1. discrete state advance (fp32, exact contract)
        const int k = safe_clip(a.env_clip[e], a.n_clips);
        const float phi = a.env_phase[e];
        const int t1 = a.env_t[e] + 1;
        const uint32_t n1 = a.env_n[e] + 1u;
        const ClipTab ci = a.clips[k];
        float phi1;
        {
#pragma clang fp contract(off)
            phi1 = phi + ci.dphi;
        }
        const bool trunc = phi1 >= 1.0f;
        int i0;
        float alpha;
        phase_index(phi1 < 1.0f ? phi1 : 1.0f, ci, &i0, &alpha);

        // 2.-3. reference FK and errors against the sim state
        const float4 *rec = a.seg + ci.seg_base + (int64_t)i0 * seg_stride(sk->B);
        float r;
        if constexpr (!MUL) {
            float e_pos = 0.0f, e_ee = 0.0f, e_vel = 0.0f;
            f3 dc = mk3(0.0f, 0.0f, 0.0f);
            auto load_pv = [&](int b) {
                SimPV s;
                s.P = ld3(a.pos, b, ld, e);
                s.V = ld3(a.linvel, b, ld, e);
                return s;
            };
            walk_prefetch<SimPV>(sk, rec, alpha, load_pv,
                                 [&](int i, int, const Frame &f, f3 A, const SimPV &sb, q4, f3) {
                const f3 dp = (sb.P - A) - f.P;
                const f3 dv = sb.V - f.V;
                const float x = dot3(dp, dp);
                e_pos += x;
                if (sk->leaf[i]) e_ee += x;
                dc = dc + sk->massw[i] * dp;
                e_vel += dot3(dv, dv);
            });
            const float e_com = dot3(dc, dc);
            r = a.c_pose * expf(-(a.w_pos * e_pos + a.w_ee * e_ee)) +
                a.c_vel * expf(-(a.w_vel * e_vel)) + a.c_com * expf(-(a.w_com * e_com));
        } else {
            MulErr me;
            walk_prefetch<SimMul>(sk, rec, alpha, [&](int b) { return load_mul(a, b, e); },
                                  [&](int i, int b, const Frame &f, f3 A, const SimMul &sb, q4 qr,
                                      f3 wr) {
                me.add(b, sk->leaf[i], sk->massw[i], f, A, sb, qr, wr);
            });
            r = me.reward(a);
        }
        const float z_root = a.pos[2 * ld + e];
        const bool term = (t1 > a.grace) && ((z_root < a.h_term) || !(r >= a.r_min));

        // 4. masked reset
        int k_out = k, t_out = t1;
        ph_out = phi1;
        if (term || trunc) {
            const uint4 x = philox4x32_10(make_uint4((uint32_t)e, n1, 0u, 1u), (uint32_t)a.seed,
                                          (uint32_t)(a.seed >> 32));
            k_out = (int)(((uint64_t)x.x * (uint64_t)(uint32_t)a.n_clips) >> 32);
            ph_out = (float)(x.y >> 8) * 0x1p-24f;
            t_out = 0;
            rsi(a, e, k_out, ph_out);
        }
        a.env_clip[e] = k_out;
        a.env_phase[e] = ph_out;
        a.env_t[e] = t_out;
        a.env_n[e] = n1;
        a.reward[e] = r;
        a.term[e] = (uint8_t)term;
        a.trunc[e] = (uint8_t)trunc;
        if (a.ref_frame) a.ref_frame[e] = i0;
        k_fin = k_out;
        reset = term || trunc;
    }
    // 5. observation of the post-reset state (this thread's own env: the
    //    reference state it may have just written is read back in order)
    if (active) {
        obs_from_sim(a, e, ph_out);
        if (a.obs_future > 0 || a.obs_prev)
            obs_extras(a, e, k_fin, ph_out, reset, sim_heading(a, e), 0, 1, a.obs_prev != 0);
    }
}

__global__ __launch_bounds__(256) void reset_kernel(EnvArgs a)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= a.n) return;
    if (a.mask && !a.mask[e]) return;
    const uint4 x = philox4x32_10(make_uint4((uint32_t)e, a.env_n[e], 0u, 4u), (uint32_t)a.seed,
                                  (uint32_t)(a.seed >> 32));
    const int k = (int)(((uint64_t)x.x * (uint64_t)(uint32_t)a.n_clips) >> 32);
    const float ph = (float)(x.y >> 8) * 0x1p-24f;
    rsi(a, e, k, ph);
    a.env_clip[e] = k;
    a.env_phase[e] = ph;
    a.env_t[e] = 0;
    obs_from_sim(a, e, ph);
    if (a.obs_future > 0 || a.obs_prev)
        obs_extras(a, e, k, ph, true, sim_heading(a, e), 0, 1, a.obs_prev != 0);
}

// ---------------------------------------------------------------------------
// Kinematic stand-in for the physics solver (benchmark and test harness).
// ---------------------------------------------------------------------------
struct NormalCache {
    uint32_t blk;
    float z[4];
};

__device__ __forceinline__ float normal_at(const EnvArgs &a, uint32_t e, uint32_t n, int j,
                                           NormalCache &nc)
{
    const uint32_t blk = (uint32_t)j >> 2;
    if (blk != nc.blk) {
        normals4(a.seed, e, n, blk, 3u, nc.z);
        nc.blk = blk;
    }
    const int q = j & 3;
    return q == 0 ? nc.z[0] : (q == 1 ? nc.z[1] : (q == 2 ? nc.z[2] : nc.z[3]));
}

__device__ __forceinline__ q4 qexp3(f3 r)
{
    const float th = sqrtf(dot3(r, r));
    if (th < 1e-20f) return q4{1.0f, 0.5f * r.x, 0.5f * r.y, 0.5f * r.z};
    float s, c;
    sincosf(0.5f * th, &s, &c);
    const float k = s / th;
    return q4{c, k * r.x, k * r.y, k * r.z};
}

struct NoisyFrame {
    Frame ref;  // noise-free reference (velocities)
    q4 Qn;      // noisy orientation
    f3 Pn;      // noisy position (anchor-relative)
};

__device__ __forceinline__ void pack_noisy(const NoisyFrame &f, float (&v)[20])
{
    float a[13];
    pack_frame(f.ref, a);
#pragma unroll
    for (int c = 0; c < 13; ++c) v[c] = a[c];
    v[13] = f.Qn.w; v[14] = f.Qn.x; v[15] = f.Qn.y; v[16] = f.Qn.z;
    v[17] = f.Pn.x; v[18] = f.Pn.y; v[19] = f.Pn.z;
}
__device__ __forceinline__ NoisyFrame unpack_noisy(const float (&v)[20])
{
    float a[13];
#pragma unroll
    for (int c = 0; c < 13; ++c) a[c] = v[c];
    NoisyFrame f;
    f.ref = unpack_frame(a);
    f.Qn = q4{v[13], v[14], v[15], v[16]};
    f.Pn = mk3(v[17], v[18], v[19]);
    return f;
}

__global__ __launch_bounds__(256) void standin_kernel(EnvArgs a)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= a.n) return;
    const int64_t ld = a.ld;
    const SkelTab *__restrict__ sk = a.sk;
    const int k = safe_clip(a.env_clip[e], a.n_clips);
    const uint32_t n = a.env_n[e];
    const ClipTab ci = a.clips[k];
    float phi1;
    {
#pragma clang fp contract(off)
        phi1 = a.env_phase[e] + ci.dphi;
    }
    int i0;
    float alpha;
    phase_index(phi1 < 1.0f ? phi1 : 1.0f, ci, &i0, &alpha);
    const float4 *rec = a.seg + ci.seg_base + (int64_t)i0 * seg_stride(sk->B);
    const float sj = a.sigma_joint, sv = a.sigma_vel;
    NormalCache nc;
    nc.blk = 0xFFFFFFFFu;
    const uint32_t ue = (uint32_t)e;
    const int zvel0 = 3 + sk->n_dof;

    auto emit = [&](int b, const NoisyFrame &f, f3 A) {
        st3(a.pos, b, ld, e, A + f.Pn);
        st4(a.quat, b, ld, e, f.Qn);
        const int jv = zvel0 + 6 * b;
        const f3 dv = mk3(normal_at(a, ue, n, jv + 0, nc), normal_at(a, ue, n, jv + 1, nc),
                          normal_at(a, ue, n, jv + 2, nc));
        const f3 dw = mk3(normal_at(a, ue, n, jv + 3, nc), normal_at(a, ue, n, jv + 4, nc),
                          normal_at(a, ue, n, jv + 5, nc));
        st3(a.linvel, b, ld, e, f.ref.V + sv * dv);
        st3(a.angvel, b, ld, e, f.ref.W + sv * dw);
    };

    const LdsStack<20> st{im_lds + threadIdx.x, (int)blockDim.x};
    float buf[20];
    f3 A;
    NoisyFrame cur;
    cur.ref = root_frame(rec, alpha, &A);
    {
        const f3 zr = mk3(normal_at(a, ue, n, 0, nc), normal_at(a, ue, n, 1, nc),
                          normal_at(a, ue, n, 2, nc));
        cur.Qn = qmul(cur.ref.Q, qexp3(sj * zr));
        cur.Pn = cur.ref.P;
    }
    emit(0, cur, A);
    if (sk->bslot[0] >= 0) {
        pack_noisy(cur, buf);
        st.put(sk->bslot[0], buf);
    }
    const int B = sk->B;
    for (int i = 1; i < B; ++i) {
        if (sk->pslot[i] >= 0) {
            st.get(sk->pslot[i], buf);
            cur = unpack_noisy(buf);
        }
        const f3 off = mk3(sk->offset[i][0], sk->offset[i][1], sk->offset[i][2]);
        const int jt = sk->jtype[i];
        const float4 *jr = rec + 6 + 3 * (i - 1);
        NoisyFrame c;
        c.ref = child_frame(cur.ref, jr, alpha, off, jt);
        q4 ql{1.0f, 0.0f, 0.0f, 0.0f};
        if (jt != IM_JOINT_FIXED) ql = slerp_basis(jr[0], jr[1], alpha * jr[2].w);
        const int jz = sk->zrot[i];
        if (jt == IM_JOINT_SPHERICAL) {
            const f3 zr = mk3(normal_at(a, ue, n, jz, nc), normal_at(a, ue, n, jz + 1, nc),
                              normal_at(a, ue, n, jz + 2, nc));
            ql = qmul(ql, qexp3(sj * zr));
        } else if (jt == IM_JOINT_REVOLUTE) {
            const float th = sj * normal_at(a, ue, n, jz, nc);
            ql = qmul(ql, qexp3(th * mk3(sk->axis[i][0], sk->axis[i][1], sk->axis[i][2])));
        }
        c.Qn = qmul(cur.Qn, ql);
        c.Pn = cur.Pn + qrot(cur.Qn, off);
        emit(sk->body[i], c, A);
        if (sk->bslot[i] >= 0) {
            pack_noisy(c, buf);
            st.put(sk->bslot[i], buf);
        }
        cur = c;
    }
}

// ---------------------------------------------------------------------------
// Creation-time packing of the reference segments (double precision).
// ---------------------------------------------------------------------------
struct dq {
    double w, x, y, z;
};

__device__ inline dq dq_norm(dq q)
{
    const double s = 1.0 / sqrt(q.w * q.w + q.x * q.x + q.y * q.y + q.z * q.z);
    return dq{q.w * s, q.x * s, q.y * s, q.z * s};
}

// rotation vector of b a^-1 (a, b unit, same hemisphere)
__device__ inline void dq_rotvec_rel(dq a, dq b, double out[3])
{
    // b (x) conj(a)
    const double w = b.w * a.w + b.x * a.x + b.y * a.y + b.z * a.z;
    const double x = -b.w * a.x + b.x * a.w - b.y * a.z + b.z * a.y;
    const double y = -b.w * a.y + b.x * a.z + b.y * a.w - b.z * a.x;
    const double z = -b.w * a.z - b.x * a.y + b.y * a.x + b.z * a.w;
    const double sgn = w < 0.0 ? -1.0 : 1.0;
    const double s = sqrt(x * x + y * y + z * z);
    if (s == 0.0) {
        out[0] = out[1] = out[2] = 0.0;
        return;
    }
    const double th = 2.0 * atan2(s, sgn * w);
    out[0] = sgn * th * x / s;
    out[1] = sgn * th * y / s;
    out[2] = sgn * th * z / s;
}

// slerp basis of (q0, q1): a, u, angle; and the constant angular velocity.
__device__ inline void basis_of(const float *q0f, const float *q1f, double fps, float4 *a_out,
                                float4 *u_out, float *ang_out, float w_out[3])
{
    const dq a = dq_norm(dq{q0f[0], q0f[1], q0f[2], q0f[3]});
    dq b = dq_norm(dq{q1f[0], q1f[1], q1f[2], q1f[3]});
    double c = a.w * b.w + a.x * b.x + a.y * b.y + a.z * b.z;
    if (c < 0.0) {
        b = dq{-b.w, -b.x, -b.y, -b.z};
        c = -c;
    }
    const double dm = sqrt((a.w - b.w) * (a.w - b.w) + (a.x - b.x) * (a.x - b.x) +
                           (a.y - b.y) * (a.y - b.y) + (a.z - b.z) * (a.z - b.z));
    const double dp = sqrt((a.w + b.w) * (a.w + b.w) + (a.x + b.x) * (a.x + b.x) +
                           (a.y + b.y) * (a.y + b.y) + (a.z + b.z) * (a.z + b.z));
    const double ang = 2.0 * atan2(dm, dp);
    dq v{b.w - c * a.w, b.x - c * a.x, b.y - c * a.y, b.z - c * a.z};
    const double vn = sqrt(v.w * v.w + v.x * v.x + v.y * v.y + v.z * v.z);
    dq u{0.0, 0.0, 0.0, 0.0};
    if (vn > 0.0) u = dq{v.w / vn, v.x / vn, v.y / vn, v.z / vn};
    *a_out = make_float4((float)a.w, (float)a.x, (float)a.y, (float)a.z);
    *u_out = make_float4((float)u.w, (float)u.x, (float)u.y, (float)u.z);
    *ang_out = (float)ang;
    double w[3];
    dq_rotvec_rel(a, b, w);
    for (int i = 0; i < 3; ++i) w_out[i] = (float)(w[i] * fps);
}

// One thread per segment i0 of one clip.
__global__ void pack_segments_kernel(const SkelTab *sk, int F, double fps,
                                     const float *root_pos, const float *root_quat,
                                     const float *local_quat, float4 *seg)
{
    const int i0 = blockIdx.x * blockDim.x + threadIdx.x;
    if (i0 >= F - 1) return;
    const int B = sk->B;
    float4 *rec = seg + (int64_t)i0 * seg_stride(B);
    const float *p0 = root_pos + 3 * i0, *p1 = root_pos + 3 * (i0 + 1);
    double d[3], v[3];
    for (int c = 0; c < 3; ++c) {
        d[c] = (double)p1[c] - (double)p0[c];
        v[c] = d[c] * fps;
    }
    float4 ra, ru;
    float ang, w[3];
    basis_of(root_quat + 4 * i0, root_quat + 4 * (i0 + 1), fps, &ra, &ru, &ang, w);
    rec[0] = make_float4(p0[0], p0[1], p0[2], (float)d[0]);
    rec[1] = make_float4((float)d[1], (float)d[2], (float)v[0], (float)v[1]);
    rec[2] = make_float4((float)v[2], w[0], w[1], w[2]);
    rec[3] = ra;
    rec[4] = ru;
    rec[5] = make_float4(ang, 0.0f, 0.0f, 0.0f);
    for (int i = 1; i < B; ++i) {
        const int b = sk->body[i];
        float4 *jr = rec + 6 + 3 * (i - 1);
        if (sk->jtype[i] == IM_JOINT_FIXED) {
            jr[0] = make_float4(1.0f, 0.0f, 0.0f, 0.0f);
            jr[1] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            jr[2] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            continue;
        }
        const float *q0 = local_quat + 4 * ((int64_t)i0 * (B - 1) + (b - 1));
        const float *q1 = local_quat + 4 * ((int64_t)(i0 + 1) * (B - 1) + (b - 1));
        basis_of(q0, q1, fps, &jr[0], &jr[1], &ang, w);
        jr[2] = make_float4(w[0], w[1], w[2], ang);
    }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called by the C ABI layer).
// ---------------------------------------------------------------------------
static hipError_t launch_env(void (*k)(EnvArgs), int n_slots, int frame_floats,
                             const EnvArgs &a, hipStream_t s)
{
    if (a.n <= 0) return hipSuccess;
    const int bs = 256;
    const size_t lds = (size_t)(n_slots > 0 ? n_slots : 1) * frame_floats * sizeof(float) * bs;
    hipLaunchKernelGGL(k, dim3((unsigned)((a.n + bs - 1) / bs)), dim3(bs), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_env_step(int n_slots, int walk_slots, const EnvArgs &a, hipStream_t s)
{
    if (a.n <= 0) return hipSuccess;
    const bool mul = a.reward_form == IM_REWARD_MULTIPLICATIVE;
    const int P = a.n_parts;
    if (P <= 1)
        return launch_env(mul ? env_step_kernel<true> : env_step_kernel<false>, n_slots, 13, a, s);
    // P threads per env: G groups of 64 envs per block of 64 P G threads; the
    // future-frame walks of the observation go over the whole skeleton (n_slots)
    const int G = P >= 4 ? 1 : 4 / P;
    const int bs = 64 * P * G;
    int slots = walk_slots;
    if (a.obs_future > 0 && n_slots > slots) slots = n_slots;
    const size_t lds = (size_t)(slots > 0 ? slots : 1) * 13 * sizeof(float) * bs;
    hipLaunchKernelGGL(mul ? env_step_parts_kernel<true> : env_step_parts_kernel<false>,
                       dim3((unsigned)((a.n + 64 * G - 1) / (64 * G))), dim3(bs), lds, s, a);
    return hipGetLastError();
}
hipError_t launch_reset(int n_slots, const EnvArgs &a, hipStream_t s)
{
    return launch_env(reset_kernel, n_slots, 13, a, s);
}
hipError_t launch_standin(int n_slots, const EnvArgs &a, hipStream_t s)
{
    return launch_env(standin_kernel, n_slots, 20, a, s);
}

hipError_t launch_pack_segments(const SkelTab *sk, int F, double fps, const float *root_pos,
                                const float *root_quat, const float *local_quat, float4 *seg,
                                hipStream_t s)
{
    const int nseg = F - 1;
    hipLaunchKernelGGL(pack_segments_kernel, dim3((nseg + 63) / 64), dim3(64), 0, s, sk, F, fps,
                       root_pos, root_quat, local_quat, seg);
    return hipGetLastError();
}

}  // namespace im
