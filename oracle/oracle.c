/*
 * oracle.c -- plain, slow CPU reference of the environment-plus-policy step
 * of GPU-native DeepMimic-style imitation training (InstantMimic, arXiv
 * 2609.09821).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or constant
 * generator with the HIP implementation.
 *
 * Precision: every continuous quantity is computed in IEEE double; outputs
 * are rounded once to float.  The discrete env state (phase, frame index,
 * counters, clip id) follows the fp32 definition below exactly (no FMA
 * contraction: build with -ffp-contract=off).
 *
 * What it computes (sections of the paper in brackets):
 *   - the rollout step of the PPO loop [Sec. 3, Fig. 3]: reward and dones
 *     are evaluated on the post-physics state, then terminated/truncated envs
 *     are reset, then the observation is built;
 *   - the tracking reward and termination flag [Sec. 4.1, Fig. 5]: body
 *     position, body velocity and centre-of-mass errors summed over bodies,
 *     exponentiated and combined, plus an end-effector position term taken
 *     from the DeepMimic reward that Sec. 6.1 builds on (weight 0 gives the
 *     printed three-term form exactly);
 *   - the unconditional reset with a device-side mask [Sec. 4.2];
 *   - heading-frame observations with the 6D rotation representation
 *     [Sec. 6.1];
 *   - the Gaussian MLP policy with a state-independent log-std [Sec. 6.1,
 *     Table "backflip config" (initial policy log std)].
 * The paper does not state how the reference clip is sampled; the reading
 * used here (linear root position, slerp rotations between the two frames
 * around the phase, exact derivatives of that path as reference velocities,
 * forward kinematics over the parent tree) is listed in the design notes.
 *
 * Parity pins live in tests/test_oracle_*.py.  Items that no pin reaches
 * (the composition of the whole step) are "parity unpinned" beyond the
 * component pins.
 *
 * Conventions: quaternions are (w,x,y,z) Hamilton [Sec. 3.2, Fig. 4a converts
 * to wxyz], active rotations, world up = +z, root forward = +x.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_MAX_BODIES 64
#define OR_JT_FREE 0
#define OR_JT_SPH 1
#define OR_JT_REV 2
#define OR_JT_FIXED 3

#define OR_TAG_ACTION 0u
#define OR_TAG_RESET 1u
#define OR_TAG_STANDIN 3u
#define OR_TAG_EXT_RESET 4u

/* ------------------------------------------------------------------ */
/* Philox4x32-10: Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: */
/* As Easy as 1, 2, 3", SC'11.  Ten rounds of the two-multiplier S-box  */
/* with the Weyl key schedule; constants from that paper.               */
/* ------------------------------------------------------------------ */
static const uint32_t PHILOX_M0 = 0xD2511F53u;
static const uint32_t PHILOX_M1 = 0xCD9E8D57u;
static const uint32_t PHILOX_W0 = 0x9E3779B9u;
static const uint32_t PHILOX_W1 = 0xBB67AE85u;

void or_philox(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)c[0];
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)c[2];
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c[1] ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c[3] ^ k1;
        uint32_t n3 = lo0;
        c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
    }
    out[0] = c[0]; out[1] = c[1]; out[2] = c[2]; out[3] = c[3];
}

static void philox_draw(uint64_t seed, uint32_t e, uint32_t n, uint32_t block, uint32_t tag,
                        uint32_t x[4])
{
    uint32_t ctr[4] = {e, n, block, tag};
    uint32_t key[2] = {(uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32)};
    or_philox(ctr, key, x);
}

/* 32-bit word -> u in (0,1): the odd multiples of 2^-24, exact in float. */
static double uniform_open(uint32_t x)
{
    return (2.0 * (double)(x >> 9) + 1.0) * 0x1p-24;
}

/* Box-Muller: (u, v) -> sqrt(-2 ln u) (cos 2 pi v, sin 2 pi v). */
void or_normals(uint64_t seed, uint32_t e, uint32_t n, uint32_t block, uint32_t tag, double z[4])
{
    uint32_t x[4];
    philox_draw(seed, e, n, block, tag, x);
    const double two_pi = 6.283185307179586476925286766559;
    for (int h = 0; h < 2; ++h) {
        double u = uniform_open(x[2 * h]);
        double v = uniform_open(x[2 * h + 1]);
        double r = sqrt(-2.0 * log(u));
        z[2 * h] = r * cos(two_pi * v);
        z[2 * h + 1] = r * sin(two_pi * v);
    }
}

/* ------------------------------------------------------------------ */
/* Quaternion and vector algebra (double).                             */
/* ------------------------------------------------------------------ */
typedef struct { double w, x, y, z; } quat;
typedef struct { double x, y, z; } vec3;

static vec3 v3(double x, double y, double z) { vec3 r = {x, y, z}; return r; }
static vec3 vadd(vec3 a, vec3 b) { return v3(a.x + b.x, a.y + b.y, a.z + b.z); }
static vec3 vsub(vec3 a, vec3 b) { return v3(a.x - b.x, a.y - b.y, a.z - b.z); }
static vec3 vscale(vec3 a, double s) { return v3(a.x * s, a.y * s, a.z * s); }
static double vdot(vec3 a, vec3 b) { return a.x * b.x + a.y * b.y + a.z * b.z; }
static vec3 vcross(vec3 a, vec3 b)
{
    return v3(a.y * b.z - a.z * b.y, a.z * b.x - a.x * b.z, a.x * b.y - a.y * b.x);
}

static quat qmake(double w, double x, double y, double z) { quat q = {w, x, y, z}; return q; }

/* Hamilton product a (x) b. */
static quat qmul(quat a, quat b)
{
    return qmake(a.w * b.w - a.x * b.x - a.y * b.y - a.z * b.z,
                 a.w * b.x + a.x * b.w + a.y * b.z - a.z * b.y,
                 a.w * b.y - a.x * b.z + a.y * b.w + a.z * b.x,
                 a.w * b.z + a.x * b.y - a.y * b.x + a.z * b.w);
}

static quat qconj(quat a) { return qmake(a.w, -a.x, -a.y, -a.z); }
static double qdot(quat a, quat b) { return a.w * b.w + a.x * b.x + a.y * b.y + a.z * b.z; }
static double qnorm(quat a) { return sqrt(qdot(a, a)); }
static quat qscale(quat a, double s) { return qmake(a.w * s, a.x * s, a.y * s, a.z * s); }
static quat qnormalize(quat a) { return qscale(a, 1.0 / qnorm(a)); }

/* Rotation matrix of the unit quaternion q/|q|, row-major. */
static void qmat(quat q, double R[9])
{
    q = qnormalize(q);
    double w = q.w, x = q.x, y = q.y, z = q.z;
    R[0] = 1.0 - 2.0 * (y * y + z * z);
    R[1] = 2.0 * (x * y - w * z);
    R[2] = 2.0 * (x * z + w * y);
    R[3] = 2.0 * (x * y + w * z);
    R[4] = 1.0 - 2.0 * (x * x + z * z);
    R[5] = 2.0 * (y * z - w * x);
    R[6] = 2.0 * (x * z - w * y);
    R[7] = 2.0 * (y * z + w * x);
    R[8] = 1.0 - 2.0 * (x * x + y * y);
}

static vec3 matvec(const double R[9], vec3 v)
{
    return v3(R[0] * v.x + R[1] * v.y + R[2] * v.z,
              R[3] * v.x + R[4] * v.y + R[5] * v.z,
              R[6] * v.x + R[7] * v.y + R[8] * v.z);
}

static vec3 qrot(quat q, vec3 v)
{
    double R[9];
    qmat(q, R);
    return matvec(R, v);
}

/* Rotation vector (log map) of q: flip to w >= 0, angle 2 atan2(|v|, w). */
static vec3 rotvec(quat q)
{
    if (q.w < 0.0) q = qscale(q, -1.0);
    double s = sqrt(q.x * q.x + q.y * q.y + q.z * q.z);
    if (s == 0.0) return v3(0.0, 0.0, 0.0);
    double theta = 2.0 * atan2(s, q.w);
    return v3(theta * q.x / s, theta * q.y / s, theta * q.z / s);
}

/* Quaternion of a rotation vector (exp map). */
static quat qexp(vec3 r)
{
    double theta = sqrt(vdot(r, r));
    if (theta == 0.0) return qmake(1.0, 0.0, 0.0, 0.0);
    double h = 0.5 * theta;
    double s = sin(h) / theta;
    return qmake(cos(h), r.x * s, r.y * s, r.z * s);
}

/*
 * Spherical linear interpolation (Shoemake 1985): flip b to a's hemisphere
 * when a.b < 0, angle Omega between the unit 4-vectors, weights
 * sin((1-t) Omega)/sin Omega and sin(t Omega)/sin Omega; linear blend when
 * sin Omega is negligible; result renormalised.
 */
static quat slerp(quat a, quat b, double t)
{
    a = qnormalize(a);
    b = qnormalize(b);
    if (qdot(a, b) < 0.0) b = qscale(b, -1.0);
    quat dm = qmake(a.w - b.w, a.x - b.x, a.y - b.y, a.z - b.z);
    quat dp = qmake(a.w + b.w, a.x + b.x, a.y + b.y, a.z + b.z);
    double omega = 2.0 * atan2(qnorm(dm), qnorm(dp));
    double so = sin(omega);
    quat q;
    if (so < 1e-12) {
        q = qmake((1.0 - t) * a.w + t * b.w, (1.0 - t) * a.x + t * b.x,
                  (1.0 - t) * a.y + t * b.y, (1.0 - t) * a.z + t * b.z);
    } else {
        double ca = sin((1.0 - t) * omega) / so;
        double cb = sin(t * omega) / so;
        q = qmake(ca * a.w + cb * b.w, ca * a.x + cb * b.x, ca * a.y + cb * b.y,
                  ca * a.z + cb * b.z);
    }
    return qnormalize(q);
}

/* Exported primitives, used by the pin tests. */
void or_qmul(const double *a, const double *b, double *out)
{
    quat r = qmul(qmake(a[0], a[1], a[2], a[3]), qmake(b[0], b[1], b[2], b[3]));
    out[0] = r.w; out[1] = r.x; out[2] = r.y; out[3] = r.z;
}
void or_qrot(const double *q, const double *v, double *out)
{
    vec3 r = qrot(qmake(q[0], q[1], q[2], q[3]), v3(v[0], v[1], v[2]));
    out[0] = r.x; out[1] = r.y; out[2] = r.z;
}
void or_rotvec(const double *q, double *out)
{
    vec3 r = rotvec(qmake(q[0], q[1], q[2], q[3]));
    out[0] = r.x; out[1] = r.y; out[2] = r.z;
}
void or_qexp(const double *r, double *out)
{
    quat q = qexp(v3(r[0], r[1], r[2]));
    out[0] = q.w; out[1] = q.x; out[2] = q.y; out[3] = q.z;
}
void or_slerp(const double *a, const double *b, double t, double *out)
{
    quat q = slerp(qmake(a[0], a[1], a[2], a[3]), qmake(b[0], b[1], b[2], b[3]), t);
    out[0] = q.w; out[1] = q.x; out[2] = q.y; out[3] = q.z;
}

/* bf16 round-to-nearest-even of a double (8 significant bits). */
static double round_bf16(double x)
{
    if (x == 0.0 || !isfinite(x)) return x;
    int ex;
    double m = frexp(x, &ex);          /* |m| in [0.5, 1) */
    double s = m * 256.0;              /* 8 significant bits above the point */
    double r = nearbyint(s);           /* default rounding mode: ties to even */
    return ldexp(r, ex - 8);
}
double or_round_bf16(double x) { return round_bf16(x); }

/* ------------------------------------------------------------------ */
/* World: skeleton, reference clips, step configuration.               */
/* ------------------------------------------------------------------ */
typedef struct {
    int F;
    double fps;
    float dphi;                 /* per-step phase increment, fp32 */
    double *root_pos;           /* [F][3] */
    double *root_quat;          /* [F][4] */
    double *local_quat;         /* [F][B-1][4] */
} or_clip;

typedef struct {
    int B;
    int parent[OR_MAX_BODIES];
    int jtype[OR_MAX_BODIES];
    int is_leaf[OR_MAX_BODIES];
    double axis[OR_MAX_BODIES][3];
    double offset[OR_MAX_BODIES][3];
    double mass[OR_MAX_BODIES];
    double total_mass;
    int n_clips;
    or_clip *clips;
    double dt;
    float h_term;
    float r_min;
    int grace;
    double c_pose, w_pos, w_ee, c_vel, w_vel, c_com, w_com;
    uint64_t seed;
    /* training terms (or_world_set_training) */
    int reward_form;            /* 0: grouped additive reward, 1: multiplicative */
    double m_w[5];              /* multiplicative weights: joint rotation, joint
                                   velocity, COM, EE position, EE orientation */
    int obs_future;             /* future reference frames in the observation */
    int obs_prev_action;        /* previous action in the observation */
    int A;                      /* action width */
    int n_ee;
    int ee[OR_MAX_BODIES];      /* end effectors (leaves) in body order */
} or_world;

/*
 * Create the world.  Arrays are the caller's float/int data:
 *   parent[B], jtype[B], axis[B*3], offset[B*3], mass[B];
 *   per clip k: F[k], fps[k]; root_pos, root_quat, local_quat concatenated
 *   over clips ([F_k][3], [F_k][4], [F_k][B-1][4]);
 *   weights[7] = c_pose, w_pos, w_ee, c_vel, w_vel, c_com, w_com.
 * Returns NULL on an inconsistent description.
 */
or_world *or_world_create(int B, const int *parent, const int *jtype, const float *axis,
                          const float *offset, const float *mass, int n_clips, const int *F,
                          const float *fps, const float *root_pos, const float *root_quat,
                          const float *local_quat, double dt, float h_term, float r_min,
                          int grace, const float *weights, uint64_t seed)
{
    if (B < 1 || B > OR_MAX_BODIES || n_clips < 1) return NULL;
    if (parent[0] != -1) return NULL;
    for (int b = 1; b < B; ++b)
        if (parent[b] < 0 || parent[b] >= b) return NULL;
    or_world *w = (or_world *)calloc(1, sizeof(or_world));
    w->B = B;
    w->total_mass = 0.0;
    for (int b = 0; b < B; ++b) {
        w->parent[b] = parent[b];
        w->jtype[b] = jtype[b];
        w->is_leaf[b] = 1;
        for (int c = 0; c < 3; ++c) {
            w->axis[b][c] = axis[3 * b + c];
            w->offset[b][c] = offset[3 * b + c];
        }
        w->mass[b] = mass[b];
        w->total_mass += mass[b];
    }
    for (int b = 1; b < B; ++b) w->is_leaf[parent[b]] = 0;
    w->n_clips = n_clips;
    w->clips = (or_clip *)calloc((size_t)n_clips, sizeof(or_clip));
    size_t rp = 0, rq = 0, lq = 0;
    for (int k = 0; k < n_clips; ++k) {
        or_clip *c = &w->clips[k];
        c->F = F[k];
        c->fps = (double)fps[k];
        if (c->F < 2) { free(w->clips); free(w); return NULL; }
        /* D1: phase increment computed once per clip in double, kept as float */
        c->dphi = (float)(dt * c->fps / (double)(c->F - 1));
        c->root_pos = (double *)malloc(sizeof(double) * 3 * (size_t)c->F);
        c->root_quat = (double *)malloc(sizeof(double) * 4 * (size_t)c->F);
        c->local_quat = (double *)malloc(sizeof(double) * 4 * (size_t)c->F * (size_t)(B > 1 ? B - 1 : 1));
        for (int i = 0; i < 3 * c->F; ++i) c->root_pos[i] = root_pos[rp + i];
        for (int i = 0; i < 4 * c->F; ++i) c->root_quat[i] = root_quat[rq + i];
        for (int i = 0; i < 4 * c->F * (B - 1); ++i) c->local_quat[i] = local_quat[lq + i];
        rp += 3 * (size_t)c->F;
        rq += 4 * (size_t)c->F;
        lq += 4 * (size_t)c->F * (size_t)(B - 1);
    }
    w->dt = dt;
    w->h_term = h_term;
    w->r_min = r_min;
    w->grace = grace;
    w->c_pose = weights[0];
    w->w_pos = weights[1];
    w->w_ee = weights[2];
    w->c_vel = weights[3];
    w->w_vel = weights[4];
    w->c_com = weights[5];
    w->w_com = weights[6];
    w->seed = seed;
    w->reward_form = 0;
    w->n_ee = 0;
    for (int b = 0; b < B; ++b)
        if (w->is_leaf[b]) w->ee[w->n_ee++] = b;
    return w;
}

/*
 * Training terms [Sec. 6.1, and the reward weights, termination and grace
 * settings of the backflip search's configuration table]:
 *   reward_form 1: r = prod_k exp(-m_k e_k) over joint rotation, joint
 *   velocity, COM, end-effector position and end-effector orientation errors;
 *   obs_future K: the reference root and end-effector frames of the next K
 *   control steps; obs_prev_action: the action applied in this step.
 */
void or_world_set_training(or_world *w, int reward_form, const float *mw, int obs_future,
                           int obs_prev_action, int A)
{
    w->reward_form = reward_form;
    for (int i = 0; i < 5; ++i) w->m_w[i] = mw[i];
    w->obs_future = obs_future;
    w->obs_prev_action = obs_prev_action;
    w->A = A;
}

/* Observation width: 15 per body, the phase, 9 per future frame of the root
 * and each end effector, and the previous action. */
int or_obs_dim(const or_world *w)
{
    return 15 * w->B + 1 + w->obs_future * (1 + w->n_ee) * 9 + (w->obs_prev_action ? w->A : 0);
}

void or_world_destroy(or_world *w)
{
    if (!w) return;
    for (int k = 0; k < w->n_clips; ++k) {
        free(w->clips[k].root_pos);
        free(w->clips[k].root_quat);
        free(w->clips[k].local_quat);
    }
    free(w->clips);
    free(w);
}

float or_clip_dphi(const or_world *w, int k) { return w->clips[k].dphi; }

/*
 * D4: evaluation phase -> frame index i0 and blend alpha, fp32 exactly:
 *   s = phi * (F-1); i0 = min(trunc(s), F-2); alpha = s - i0.
 */
void or_phase_index(int F, float phi_ev, int *i0_out, float *alpha_out)
{
    float s = phi_ev * (float)(F - 1);
    int i0 = (int)s;
    if (i0 > F - 2) i0 = F - 2;
    float alpha = s - (float)i0;
    *i0_out = i0;
    *alpha_out = alpha;
}

/* A pose in local (joint) coordinates plus the root's world motion. */
typedef struct {
    vec3 root_p, root_v, root_w;
    quat root_q;
    quat q[OR_MAX_BODIES];      /* local rotation of body b in its parent frame */
    vec3 wrel[OR_MAX_BODIES];   /* local angular velocity, parent frame */
} or_local;

/* World-frame body state. */
typedef struct {
    vec3 P[OR_MAX_BODIES], V[OR_MAX_BODIES], W[OR_MAX_BODIES];
    quat Q[OR_MAX_BODIES];
} or_state;

static quat clip_root_q(const or_clip *c, int i)
{
    const double *r = c->root_quat + 4 * i;
    return qmake(r[0], r[1], r[2], r[3]);
}
static vec3 clip_root_p(const or_clip *c, int i)
{
    const double *r = c->root_pos + 3 * i;
    return v3(r[0], r[1], r[2]);
}
static quat clip_local_q(const or_world *w, const or_clip *c, int i, int b)
{
    const double *r = c->local_quat + 4 * ((size_t)i * (size_t)(w->B - 1) + (size_t)(b - 1));
    return qmake(r[0], r[1], r[2], r[3]);
}

/*
 * Reference pose at clip k between frames i0 and i0+1 with blend alpha:
 * linear root position, slerped root and joint rotations; the velocities are
 * the exact time derivatives of that path inside the segment (the blend
 * advances at fps per second):
 *   root v = (P1 - P0) fps,  root w = rotvec(Q1 Q0^-1) fps  (world),
 *   joint w = rotvec(q1 q0^-1) fps                          (parent frame).
 */
static void ref_local(const or_world *w, int k, int i0, double alpha, or_local *L)
{
    const or_clip *c = &w->clips[k];
    vec3 p0 = clip_root_p(c, i0), p1 = clip_root_p(c, i0 + 1);
    quat q0 = clip_root_q(c, i0), q1 = clip_root_q(c, i0 + 1);
    L->root_p = vadd(vscale(p0, 1.0 - alpha), vscale(p1, alpha));
    L->root_q = slerp(q0, q1, alpha);
    L->root_v = vscale(vsub(p1, p0), c->fps);
    L->root_w = vscale(rotvec(qmul(q1, qconj(q0))), c->fps);
    L->q[0] = qmake(1.0, 0.0, 0.0, 0.0);
    L->wrel[0] = v3(0.0, 0.0, 0.0);
    for (int b = 1; b < w->B; ++b) {
        if (w->jtype[b] == OR_JT_FIXED) {
            L->q[b] = qmake(1.0, 0.0, 0.0, 0.0);
            L->wrel[b] = v3(0.0, 0.0, 0.0);
            continue;
        }
        quat a = clip_local_q(w, c, i0, b), bq = clip_local_q(w, c, i0 + 1, b);
        L->q[b] = slerp(a, bq, alpha);
        L->wrel[b] = vscale(rotvec(qmul(bq, qconj(a))), c->fps);
    }
}

/*
 * Forward kinematics in body index order (parent[b] < b):
 *   Q_b = Q_p q_b,  P_b = P_p + R(Q_p) offset_b,
 *   W_b = W_p + R(Q_p) wrel_b,  V_b = V_p + W_p x (P_b - P_p).
 */
static void fk(const or_world *w, const or_local *L, or_state *S)
{
    S->P[0] = L->root_p;
    S->Q[0] = L->root_q;
    S->V[0] = L->root_v;
    S->W[0] = L->root_w;
    for (int b = 1; b < w->B; ++b) {
        int p = w->parent[b];
        double R[9];
        qmat(S->Q[p], R);
        vec3 off = v3(w->offset[b][0], w->offset[b][1], w->offset[b][2]);
        S->Q[b] = qmul(S->Q[p], L->q[b]);
        S->P[b] = vadd(S->P[p], matvec(R, off));
        S->W[b] = vadd(S->W[p], matvec(R, L->wrel[b]));
        S->V[b] = vadd(S->V[p], vcross(S->W[p], vsub(S->P[b], S->P[p])));
    }
}

static void ref_state(const or_world *w, int k, float phi_ev, or_state *S)
{
    int i0;
    float alpha;
    or_phase_index(w->clips[k].F, phi_ev, &i0, &alpha);
    or_local L;
    ref_local(w, k, i0, (double)alpha, &L);
    fk(w, &L, S);
}

/* Exported: reference world state of clip k at evaluation phase phi_ev. */
void or_ref_state(const or_world *w, int k, float phi_ev, double *P, double *Q, double *V,
                  double *W)
{
    or_state S;
    ref_state(w, k, phi_ev, &S);
    for (int b = 0; b < w->B; ++b) {
        P[3 * b] = S.P[b].x; P[3 * b + 1] = S.P[b].y; P[3 * b + 2] = S.P[b].z;
        Q[4 * b] = S.Q[b].w; Q[4 * b + 1] = S.Q[b].x; Q[4 * b + 2] = S.Q[b].y; Q[4 * b + 3] = S.Q[b].z;
        V[3 * b] = S.V[b].x; V[3 * b + 1] = S.V[b].y; V[3 * b + 2] = S.V[b].z;
        W[3 * b] = S.W[b].x; W[3 * b + 1] = S.W[b].y; W[3 * b + 2] = S.W[b].z;
    }
}

/* Exported: FK of an arbitrary local pose (pins).  q_local [B][4] (row 0
 * ignored), w_local [B][3]; root p/q/v/w given. */
void or_fk(const or_world *w, const double *root_p, const double *root_q, const double *root_v,
           const double *root_w, const double *q_local, const double *w_local, double *P,
           double *Q, double *V, double *W)
{
    or_local L;
    L.root_p = v3(root_p[0], root_p[1], root_p[2]);
    L.root_q = qmake(root_q[0], root_q[1], root_q[2], root_q[3]);
    L.root_v = v3(root_v[0], root_v[1], root_v[2]);
    L.root_w = v3(root_w[0], root_w[1], root_w[2]);
    for (int b = 0; b < w->B; ++b) {
        L.q[b] = qmake(q_local[4 * b], q_local[4 * b + 1], q_local[4 * b + 2], q_local[4 * b + 3]);
        L.wrel[b] = v3(w_local[3 * b], w_local[3 * b + 1], w_local[3 * b + 2]);
    }
    or_state S;
    fk(w, &L, &S);
    for (int b = 0; b < w->B; ++b) {
        P[3 * b] = S.P[b].x; P[3 * b + 1] = S.P[b].y; P[3 * b + 2] = S.P[b].z;
        Q[4 * b] = S.Q[b].w; Q[4 * b + 1] = S.Q[b].x; Q[4 * b + 2] = S.Q[b].y; Q[4 * b + 3] = S.Q[b].z;
        V[3 * b] = S.V[b].x; V[3 * b + 1] = S.V[b].y; V[3 * b + 2] = S.V[b].z;
        W[3 * b] = S.W[b].x; W[3 * b + 1] = S.W[b].y; W[3 * b + 2] = S.W[b].z;
    }
}

/* ------------------------------------------------------------------ */
/* Reward [Sec. 4.1, Fig. 5] with the end-effector term.               */
/* ------------------------------------------------------------------ */
typedef struct { double e_pos, e_vel, e_ee, e_com, r; } or_reward_t;

/*
 * Errors are sums over bodies of squared distances (Fig. 5 sums over the
 * body and coordinate axes): e_pos over all bodies' positions, e_vel over
 * their linear velocities, e_ee over end effectors (bodies without
 * children), e_com on the mass-weighted centre of body origins.
 *   r = c_pose exp(-(w_pos e_pos + w_ee e_ee)) + c_vel exp(-w_vel e_vel)
 *       + c_com exp(-w_com e_com)
 */
static or_reward_t reward_of(const or_world *w, const vec3 *P, const vec3 *V, const vec3 *Pr,
                             const vec3 *Vr)
{
    or_reward_t out = {0, 0, 0, 0, 0};
    vec3 c = v3(0, 0, 0), cr = v3(0, 0, 0);
    for (int b = 0; b < w->B; ++b) {
        vec3 dp = vsub(P[b], Pr[b]);
        vec3 dv = vsub(V[b], Vr[b]);
        out.e_pos += vdot(dp, dp);
        out.e_vel += vdot(dv, dv);
        if (w->is_leaf[b]) out.e_ee += vdot(dp, dp);
        c = vadd(c, vscale(P[b], w->mass[b]));
        cr = vadd(cr, vscale(Pr[b], w->mass[b]));
    }
    c = vscale(c, 1.0 / w->total_mass);
    cr = vscale(cr, 1.0 / w->total_mass);
    vec3 dc = vsub(c, cr);
    out.e_com = vdot(dc, dc);
    out.r = w->c_pose * exp(-(w->w_pos * out.e_pos + w->w_ee * out.e_ee)) +
            w->c_vel * exp(-w->w_vel * out.e_vel) + w->c_com * exp(-w->w_com * out.e_com);
    return out;
}

/* Exported for pins: P, V, Pr, Vr as [B][3] doubles; out = e_pos, e_vel,
 * e_ee, e_com, r (double). */
void or_reward(const or_world *w, const double *P, const double *V, const double *Pr,
               const double *Vr, double *out)
{
    vec3 a[OR_MAX_BODIES], bv[OR_MAX_BODIES], c[OR_MAX_BODIES], d[OR_MAX_BODIES];
    for (int b = 0; b < w->B; ++b) {
        a[b] = v3(P[3 * b], P[3 * b + 1], P[3 * b + 2]);
        bv[b] = v3(V[3 * b], V[3 * b + 1], V[3 * b + 2]);
        c[b] = v3(Pr[3 * b], Pr[3 * b + 1], Pr[3 * b + 2]);
        d[b] = v3(Vr[3 * b], Vr[3 * b + 1], Vr[3 * b + 2]);
    }
    or_reward_t r = reward_of(w, a, bv, c, d);
    out[0] = r.e_pos; out[1] = r.e_vel; out[2] = r.e_ee; out[3] = r.e_com; out[4] = r.r;
}

/* Rotation angle in [0, pi] of a unit quaternion (either sign). */
static double qangle(quat q)
{
    double v = sqrt(q.x * q.x + q.y * q.y + q.z * q.z);
    return 2.0 * atan2(v, fabs(q.w));
}

typedef struct { double e_jrot, e_jvel, e_com, e_eepos, e_eerot, r; } or_mreward_t;

/*
 * Multiplicative imitation reward [Sec. 6.1]: r = prod_k exp(-m_k e_k) with
 *   e_jrot  = sum_b angle(qr_b^-1 q_b)^2, q_b the joint rotation (parent frame;
 *             the root's world orientation for b = 0), qr_b the reference's;
 *   e_jvel  = sum_b |w_b - wr_b|^2, w_b the joint angular velocity in the parent
 *             frame, R(Q_p)^T (W_b - W_p) (the root's world angular velocity);
 *   e_com   = |c - cr|^2 (point masses at body origins);
 *   e_eepos = sum_e |P_e - Pr_e|^2 over end effectors;
 *   e_eerot = sum_e angle(Qr_e^-1 Q_e)^2 (world orientations).
 */
static or_mreward_t mreward_of(const or_world *w, const vec3 *P, const quat *Q, const vec3 *W,
                               const or_local *L, const or_state *Sr)
{
    or_mreward_t out = {0, 0, 0, 0, 0, 0};
    vec3 c = v3(0, 0, 0), cr = v3(0, 0, 0);
    for (int b = 0; b < w->B; ++b) {
        quat ql, qr;
        vec3 wl, wr;
        if (b == 0) {
            ql = Q[0];
            qr = L->root_q;
            wl = W[0];
            wr = L->root_w;
        } else {
            int p = w->parent[b];
            ql = qmul(qconj(Q[p]), Q[b]);
            qr = L->q[b];
            wl = qrot(qconj(Q[p]), vsub(W[b], W[p]));
            wr = L->wrel[b];
        }
        double th = qangle(qmul(qconj(qr), ql));
        out.e_jrot += th * th;
        vec3 dw = vsub(wl, wr);
        out.e_jvel += vdot(dw, dw);
        c = vadd(c, vscale(P[b], w->mass[b]));
        cr = vadd(cr, vscale(Sr->P[b], w->mass[b]));
        if (w->is_leaf[b]) {
            vec3 dp = vsub(P[b], Sr->P[b]);
            out.e_eepos += vdot(dp, dp);
            double te = qangle(qmul(qconj(Sr->Q[b]), Q[b]));
            out.e_eerot += te * te;
        }
    }
    c = vscale(c, 1.0 / w->total_mass);
    cr = vscale(cr, 1.0 / w->total_mass);
    vec3 dc = vsub(c, cr);
    out.e_com = vdot(dc, dc);
    out.r = exp(-w->m_w[0] * out.e_jrot) * exp(-w->m_w[1] * out.e_jvel) *
            exp(-w->m_w[2] * out.e_com) * exp(-w->m_w[3] * out.e_eepos) *
            exp(-w->m_w[4] * out.e_eerot);
    return out;
}

/* Exported for pins: the sim state as doubles ([B][3], [B][4], ...) against the
 * reference of clip k at phase phi_ev; out = e_jrot, e_jvel, e_com, e_eepos,
 * e_eerot, r. */
void or_mreward(const or_world *w, const double *P, const double *Q, const double *W, int k,
                float phi_ev, double *out)
{
    vec3 a[OR_MAX_BODIES], c[OR_MAX_BODIES];
    quat q[OR_MAX_BODIES];
    for (int b = 0; b < w->B; ++b) {
        a[b] = v3(P[3 * b], P[3 * b + 1], P[3 * b + 2]);
        q[b] = qmake(Q[4 * b], Q[4 * b + 1], Q[4 * b + 2], Q[4 * b + 3]);
        c[b] = v3(W[3 * b], W[3 * b + 1], W[3 * b + 2]);
    }
    int i0;
    float alpha;
    or_phase_index(w->clips[k].F, phi_ev, &i0, &alpha);
    or_local L;
    ref_local(w, k, i0, (double)alpha, &L);
    or_state Sr;
    fk(w, &L, &Sr);
    or_mreward_t r = mreward_of(w, a, q, c, &L, &Sr);
    out[0] = r.e_jrot; out[1] = r.e_jvel; out[2] = r.e_com; out[3] = r.e_eepos;
    out[4] = r.e_eerot; out[5] = r.r;
}

/*
 * Termination [Fig. 5, strict "<"]: after the grace steps, an env
 * terminates when the root is below h_term or the fp32 reward is not at
 * least r_min (a NaN reward terminates).
 */
static int terminated_of(const or_world *w, int t_next, float z_root, float r_out)
{
    if (!(t_next > w->grace)) return 0;
    return (z_root < w->h_term) || !(r_out >= w->r_min);
}

int or_terminated(const or_world *w, int t_next, float z_root, float r_out)
{
    return terminated_of(w, t_next, z_root, r_out);
}

/* ------------------------------------------------------------------ */
/* Sim-state access, SoA [B][comp][ld] floats.                         */
/* ------------------------------------------------------------------ */
typedef struct {
    float *pos, *quat, *linvel, *angvel;
    int64_t ld;
} or_sim;

static vec3 sim_v3(const float *a, int b, int64_t ld, int64_t e)
{
    return v3(a[(3 * (int64_t)b + 0) * ld + e], a[(3 * (int64_t)b + 1) * ld + e],
              a[(3 * (int64_t)b + 2) * ld + e]);
}
static quat sim_q(const float *a, int b, int64_t ld, int64_t e)
{
    return qmake(a[(4 * (int64_t)b + 0) * ld + e], a[(4 * (int64_t)b + 1) * ld + e],
                 a[(4 * (int64_t)b + 2) * ld + e], a[(4 * (int64_t)b + 3) * ld + e]);
}
static void put_v3(float *a, int b, int64_t ld, int64_t e, vec3 v)
{
    a[(3 * (int64_t)b + 0) * ld + e] = (float)v.x;
    a[(3 * (int64_t)b + 1) * ld + e] = (float)v.y;
    a[(3 * (int64_t)b + 2) * ld + e] = (float)v.z;
}
static void put_q(float *a, int b, int64_t ld, int64_t e, quat q)
{
    a[(4 * (int64_t)b + 0) * ld + e] = (float)q.w;
    a[(4 * (int64_t)b + 1) * ld + e] = (float)q.x;
    a[(4 * (int64_t)b + 2) * ld + e] = (float)q.y;
    a[(4 * (int64_t)b + 3) * ld + e] = (float)q.z;
}

static void write_state(const or_world *w, const or_sim *s, int64_t e, const or_state *S)
{
    for (int b = 0; b < w->B; ++b) {
        put_v3(s->pos, b, s->ld, e, S->P[b]);
        put_q(s->quat, b, s->ld, e, S->Q[b]);
        put_v3(s->linvel, b, s->ld, e, S->V[b]);
        put_v3(s->angvel, b, s->ld, e, S->W[b]);
    }
}

/* ------------------------------------------------------------------ */
/* Observation [Sec. 6.1]: heading frame, 6D rotations.                */
/* ------------------------------------------------------------------ */
/*
 * Heading: the root's forward axis f = R(Q_0) x projected on the ground
 * plane, (c, s) = (f_x, f_y)/|(f_x, f_y)| (identity if degenerate).
 * H^T rotates world vectors by -yaw about z; o = (P_0x, P_0y, 0).
 * Per body b, 15 floats: H^T (P_b - o); the first two columns of
 * H^T R(Q_b) as (M00, M10, M20, M01, M11, M21) [6D representation of Zhou
 * et al. cited in Sec. 6.1]; H^T V_b; H^T W_b.  Last entry: the phase.
 */
/* H^T of the heading frame of root orientation Q0 (identity if degenerate). */
static void heading_T(quat Q0, double HT[9])
{
    double R0[9];
    qmat(Q0, R0);
    double fx = R0[0], fy = R0[3];
    double h2 = fx * fx + fy * fy;
    double c = 1.0, s = 0.0;
    if (!(h2 < 1e-12)) {
        double hn = sqrt(h2);
        c = fx / hn;
        s = fy / hn;
    }
    double M[9] = {c, s, 0.0, -s, c, 0.0, 0.0, 0.0, 1.0};
    for (int i = 0; i < 9; ++i) HT[i] = M[i];
}

/* 9 values of a frame in the heading frame: H^T (P - o), then the first two
 * columns of H^T R(Q). */
static void frame9(const double HT[9], vec3 org, vec3 P, quat Q, double *o)
{
    vec3 p = matvec(HT, vsub(P, org));
    double R[9];
    qmat(Q, R);
    vec3 col0 = matvec(HT, v3(R[0], R[3], R[6]));
    vec3 col1 = matvec(HT, v3(R[1], R[4], R[7]));
    o[0] = p.x; o[1] = p.y; o[2] = p.z;
    o[3] = col0.x; o[4] = col0.y; o[5] = col0.z;
    o[6] = col1.x; o[7] = col1.y; o[8] = col1.z;
}

static void obs_of(const or_world *w, const vec3 *P, const quat *Q, const vec3 *V,
                   const vec3 *W, float phase, double *o_out)
{
    double HT[9];
    heading_T(Q[0], HT);
    vec3 org = v3(P[0].x, P[0].y, 0.0);
    for (int b = 0; b < w->B; ++b) {
        double *o = o_out + 15 * b;
        frame9(HT, org, P[b], Q[b], o);
        vec3 lv = matvec(HT, V[b]);
        vec3 av = matvec(HT, W[b]);
        o[9] = lv.x; o[10] = lv.y; o[11] = lv.z;
        o[12] = av.x; o[13] = av.y; o[14] = av.z;
    }
    o_out[15 * w->B] = (double)phase;
}

/*
 * Observation extras after the 15B+1 rows [Sec. 6.1, PHC observation]: for
 * j = 1..K the reference of clip k at the phase of the j-th next control
 * step (ph_j = ph_{j-1} + dphi_k in fp32, evaluated at min(ph_j, 1)): the
 * root, then each end effector in body order, as 9 values in the heading
 * frame of the current sim root; then the previous action (zeros for NULL).
 */
static void obs_extras(const or_world *w, int k, float ph, quat Q0, vec3 P0, const float *prev,
                       double *o)
{
    double HT[9];
    heading_T(Q0, HT);
    vec3 org = v3(P0.x, P0.y, 0.0);
    int idx = 0;
    float phj = ph;
    for (int j = 1; j <= w->obs_future; ++j) {
        phj = phj + w->clips[k].dphi;
        float phi_ev = phj < 1.0f ? phj : 1.0f;
        or_state S;
        ref_state(w, k, phi_ev, &S);
        for (int m = 0; m <= w->n_ee; ++m) {
            int b = m == 0 ? 0 : w->ee[m - 1];
            frame9(HT, org, S.P[b], S.Q[b], o + idx);
            idx += 9;
        }
    }
    if (w->obs_prev_action)
        for (int a = 0; a < w->A; ++a) o[idx++] = prev ? (double)prev[a] : 0.0;
}

static void obs_from_sim(const or_world *w, const or_sim *s, int64_t e, float phase, int k,
                         const float *prev, float *obs, int64_t ld_obs)
{
    vec3 P[OR_MAX_BODIES], V[OR_MAX_BODIES], W[OR_MAX_BODIES];
    quat Q[OR_MAX_BODIES];
    for (int b = 0; b < w->B; ++b) {
        P[b] = sim_v3(s->pos, b, s->ld, e);
        Q[b] = sim_q(s->quat, b, s->ld, e);
        V[b] = sim_v3(s->linvel, b, s->ld, e);
        W[b] = sim_v3(s->angvel, b, s->ld, e);
    }
    double o[15 * OR_MAX_BODIES + 1 + 4 * (OR_MAX_BODIES + 1) * 9 + 256];
    obs_of(w, P, Q, V, W, phase, o);
    int D0 = 15 * w->B + 1;
    obs_extras(w, k, phase, Q[0], P[0], prev, o + D0);
    int D = or_obs_dim(w);
    for (int i = 0; i < D; ++i) obs[(int64_t)i * ld_obs + e] = (float)o[i];
}

/* Exported for pins: one env's state as doubles ([B][3], [B][4], ...). */
void or_obs(const or_world *w, const double *P, const double *Q, const double *V, const double *W,
            float phase, double *out)
{
    vec3 a[OR_MAX_BODIES], c[OR_MAX_BODIES], d[OR_MAX_BODIES];
    quat q[OR_MAX_BODIES];
    for (int b = 0; b < w->B; ++b) {
        a[b] = v3(P[3 * b], P[3 * b + 1], P[3 * b + 2]);
        q[b] = qmake(Q[4 * b], Q[4 * b + 1], Q[4 * b + 2], Q[4 * b + 3]);
        c[b] = v3(V[3 * b], V[3 * b + 1], V[3 * b + 2]);
        d[b] = v3(W[3 * b], W[3 * b + 1], W[3 * b + 2]);
    }
    obs_of(w, a, q, c, d, phase, out);
}

/* ------------------------------------------------------------------ */
/* Reset draw: uniform clip and uniform phase in [0, 1).               */
/* ------------------------------------------------------------------ */
void or_reset_draw(const or_world *w, uint32_t e, uint32_t n, uint32_t tag, int *k_out,
                   float *phi_out)
{
    uint32_t x[4];
    philox_draw(w->seed, e, n, 0u, tag, x);
    *k_out = (int)(((uint64_t)x[0] * (uint64_t)w->n_clips) >> 32);
    *phi_out = (float)(x[1] >> 8) * 0x1p-24f;
}

/* Reset one env to the reference state (RSI) at a fresh (clip, phase). */
static void reset_one(const or_world *w, const or_sim *s, int64_t e, uint32_t n, uint32_t tag,
                      int32_t *env_clip, float *env_phase, int32_t *env_t)
{
    int k;
    float phi;
    or_reset_draw(w, (uint32_t)e, n, tag, &k, &phi);
    env_clip[e] = k;
    env_phase[e] = phi;
    env_t[e] = 0;
    or_state S;
    ref_state(w, k, phi, &S);
    write_state(w, s, e, &S);
}

/* ------------------------------------------------------------------ */
/* The fused environment step, per env.                                */
/* ------------------------------------------------------------------ */
static void env_step_one(const or_world *w, int64_t e, int32_t *env_clip, float *env_phase,
                         int32_t *env_t, uint32_t *env_n, const or_sim *s, float *reward,
                         uint8_t *term_out, uint8_t *trunc_out, float *obs, int64_t ld_obs,
                         int32_t *ref_frame, const float *prev_action)
{
    int k = env_clip[e];
    const or_clip *c = &w->clips[k];
    /* D2/D3: phase, step and counter advance; truncation at the clip end */
    float phi1 = env_phase[e] + c->dphi;
    int t1 = env_t[e] + 1;
    uint32_t n1 = env_n[e] + 1u;
    int trunc = (phi1 >= 1.0f);
    float phi_ev = phi1 < 1.0f ? phi1 : 1.0f;
    int i0;
    float alpha;
    or_phase_index(c->F, phi_ev, &i0, &alpha);
    if (ref_frame) ref_frame[e] = i0;

    /* reference at the new phase, sim state as given by the physics */
    or_local L;
    ref_local(w, k, i0, (double)alpha, &L);
    or_state Sr;
    fk(w, &L, &Sr);
    vec3 P[OR_MAX_BODIES], V[OR_MAX_BODIES], W[OR_MAX_BODIES];
    quat Q[OR_MAX_BODIES];
    for (int b = 0; b < w->B; ++b) {
        P[b] = sim_v3(s->pos, b, s->ld, e);
        V[b] = sim_v3(s->linvel, b, s->ld, e);
        Q[b] = sim_q(s->quat, b, s->ld, e);
        W[b] = sim_v3(s->angvel, b, s->ld, e);
    }
    float r_out;
    if (w->reward_form == 1) {
        or_mreward_t r = mreward_of(w, P, Q, W, &L, &Sr);
        r_out = (float)r.r;
    } else {
        or_reward_t r = reward_of(w, P, V, Sr.P, Sr.V);
        r_out = (float)r.r;
    }
    float z_root = s->pos[2 * s->ld + e];
    int term = terminated_of(w, t1, z_root, r_out);
    reward[e] = r_out;
    term_out[e] = (uint8_t)term;
    trunc_out[e] = (uint8_t)trunc;

    /* masked reset (every env runs this; only done envs change) */
    env_n[e] = n1;
    const float *prev = NULL;
    if (term || trunc) {
        reset_one(w, s, e, n1, OR_TAG_RESET, env_clip, env_phase, env_t);
    } else {
        env_phase[e] = phi1;
        env_t[e] = t1;
        if (w->obs_prev_action && prev_action) prev = prev_action + (int64_t)w->A * e;
    }
    /* observation of the post-reset state (a reset env has no previous action) */
    obs_from_sim(w, s, e, env_phase[e], env_clip[e], prev, obs, ld_obs);
}

/*
 * Batch step over envs idx[0..n_idx) (all N envs when idx is NULL).
 * Buffers follow the library's layout: env arrays [ld], sim [B][c][ld],
 * outputs [ld], obs [D][ld_obs] (D = or_obs_dim).  ref_frame may be NULL;
 * prev_action ([N][A], the actions applied in this step) may be NULL when the
 * observation has no previous-action rows.
 */
void or_env_step(const or_world *w, int64_t N, const int64_t *idx, int64_t n_idx,
                 int32_t *env_clip, float *env_phase, int32_t *env_t, uint32_t *env_n,
                 float *pos, float *quat_, float *linvel, float *angvel, int64_t ld,
                 float *reward, uint8_t *term, uint8_t *trunc, float *obs, int64_t ld_obs,
                 int32_t *ref_frame, const float *prev_action)
{
    or_sim s = {pos, quat_, linvel, angvel, ld};
    int64_t m = idx ? n_idx : N;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < m; ++j) {
        int64_t e = idx ? idx[j] : j;
        env_step_one(w, e, env_clip, env_phase, env_t, env_n, &s, reward, term, trunc, obs,
                     ld_obs, ref_frame, prev_action);
    }
}

/*
 * Host- or start-forced reset of the envs whose mask byte is non-zero (all
 * envs when mask is NULL).  Draws with the external-reset tag at the env's
 * current counter; the counter is not advanced.  Writes env state, RSI sim
 * state and the observation.
 */
void or_reset_envs(const or_world *w, int64_t N, const uint8_t *mask, int32_t *env_clip,
                   float *env_phase, int32_t *env_t, uint32_t *env_n, float *pos, float *quat_,
                   float *linvel, float *angvel, int64_t ld, float *obs, int64_t ld_obs)
{
    or_sim s = {pos, quat_, linvel, angvel, ld};
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < N; ++e) {
        if (mask && !mask[e]) continue;
        reset_one(w, &s, e, env_n[e], OR_TAG_EXT_RESET, env_clip, env_phase, env_t);
        obs_from_sim(w, &s, e, env_phase[e], env_clip[e], NULL, obs, ld_obs);
    }
}

/* ------------------------------------------------------------------ */
/* Kinematic stand-in for the physics solver (harness input).          */
/* ------------------------------------------------------------------ */
/*
 * Sim state for the step about to be evaluated: the reference at the env's
 * next phase with Gaussian rotation noise composed on the right of the root
 * orientation and of every non-fixed joint (3 DoF spherical, 1 DoF about the
 * axis for revolute), root position exact, and velocities equal to the
 * reference ones plus Gaussian noise.  Normal j comes from Philox block
 * j/4, lane j%4, tag 3, counter (e, n).  Order: root rotation (3); per
 * body 1..B-1 its DoFs; then per body 0..B-1 linear (3) and angular (3)
 * velocity.
 */
static void standin_one(const or_world *w, int64_t e, const int32_t *env_clip,
                        const float *env_phase, const uint32_t *env_n, double sig_j,
                        double sig_v, const or_sim *s)
{
    int k = env_clip[e];
    const or_clip *c = &w->clips[k];
    float phi1 = env_phase[e] + c->dphi;
    float phi_ev = phi1 < 1.0f ? phi1 : 1.0f;
    int i0;
    float alpha;
    or_phase_index(c->F, phi_ev, &i0, &alpha);
    or_local L;
    ref_local(w, k, i0, (double)alpha, &L);
    or_state Sr;
    fk(w, &L, &Sr);

    int nz = 3;
    for (int b = 1; b < w->B; ++b)
        nz += (w->jtype[b] == OR_JT_SPH) ? 3 : (w->jtype[b] == OR_JT_REV ? 1 : 0);
    nz += 6 * w->B;
    double z[4 * (6 * OR_MAX_BODIES + 3 * OR_MAX_BODIES + 4) / 4 + 8];
    for (int m = 0; 4 * m < nz; ++m)
        or_normals(w->seed, (uint32_t)e, env_n[e], (uint32_t)m, OR_TAG_STANDIN, z + 4 * m);

    int j = 0;
    or_local Ln = L;
    Ln.root_q = qmul(L.root_q, qexp(v3(sig_j * z[0], sig_j * z[1], sig_j * z[2])));
    j = 3;
    for (int b = 1; b < w->B; ++b) {
        if (w->jtype[b] == OR_JT_SPH) {
            Ln.q[b] = qmul(L.q[b], qexp(v3(sig_j * z[j], sig_j * z[j + 1], sig_j * z[j + 2])));
            j += 3;
        } else if (w->jtype[b] == OR_JT_REV) {
            double a = sig_j * z[j];
            Ln.q[b] = qmul(L.q[b], qexp(v3(a * w->axis[b][0], a * w->axis[b][1], a * w->axis[b][2])));
            j += 1;
        }
    }
    or_state Sn;
    fk(w, &Ln, &Sn);
    for (int b = 0; b < w->B; ++b) {
        Sn.V[b] = vadd(Sr.V[b], v3(sig_v * z[j], sig_v * z[j + 1], sig_v * z[j + 2]));
        Sn.W[b] = vadd(Sr.W[b], v3(sig_v * z[j + 3], sig_v * z[j + 4], sig_v * z[j + 5]));
        j += 6;
    }
    write_state(w, s, e, &Sn);
}

void or_standin(const or_world *w, int64_t N, const int64_t *idx, int64_t n_idx,
                const int32_t *env_clip, const float *env_phase, const uint32_t *env_n,
                float sigma_joint, float sigma_vel, float *pos, float *quat_, float *linvel,
                float *angvel, int64_t ld)
{
    or_sim s = {pos, quat_, linvel, angvel, ld};
    int64_t m = idx ? n_idx : N;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < m; ++j) {
        int64_t e = idx ? idx[j] : j;
        standin_one(w, e, env_clip, env_phase, env_n, (double)sigma_joint, (double)sigma_vel, &s);
    }
}

/* ------------------------------------------------------------------ */
/* Gaussian MLP policy [Sec. 3 Fig. 3 "policy(obs)", Sec. 6.1].        */
/* ------------------------------------------------------------------ */
/*
 * dims[0..L]: dims[0] = observation width, dims[L] = action width.
 * W: concatenated W_l [dims[l+1]][dims[l]] (nn.Linear order), b likewise.
 * bf16 != 0: the input and every hidden activation are rounded to bf16
 * (weights are given already bf16-valued); accumulation is double.
 * Hidden layers use ReLU; the last layer is linear and gives the mean.
 * Actions: a = mu + exp(log_std) z with z from Philox tag 0, counter
 * (e, n, j) for the block j of four actions, Box-Muller;
 * logp = -sum(z^2/2 + log_std + ln(2 pi)/2).
 */
void or_policy(int L, const int *dims, int bf16, const float *Wall, const float *ball,
               const float *log_std, uint64_t seed, int64_t N, const float *obs, int64_t ld_obs,
               const uint32_t *env_n, const int64_t *idx, int64_t n_idx, float *mean,
               float *action, float *logp)
{
    int maxw = 0;
    for (int l = 0; l <= L; ++l) maxw = dims[l] > maxw ? dims[l] : maxw;
    int64_t m = idx ? n_idx : N;
    const int A = dims[L];
    const double half_log_2pi = 0.91893853320467274178032973640562;
#pragma omp parallel
    {
        double *h = (double *)malloc(sizeof(double) * (size_t)maxw);
        double *y = (double *)malloc(sizeof(double) * (size_t)maxw);
#pragma omp for schedule(static)
        for (int64_t jj = 0; jj < m; ++jj) {
            int64_t e = idx ? idx[jj] : jj;
            for (int i = 0; i < dims[0]; ++i) {
                double x = (double)obs[(int64_t)i * ld_obs + e];
                h[i] = bf16 ? round_bf16(x) : x;
            }
            size_t woff = 0, boff = 0;
            for (int l = 0; l < L; ++l) {
                int nin = dims[l], nout = dims[l + 1];
                for (int o = 0; o < nout; ++o) {
                    double acc = 0.0;
                    const float *wr = Wall + woff + (size_t)o * (size_t)nin;
                    for (int i = 0; i < nin; ++i) acc += (double)wr[i] * h[i];
                    acc += (double)ball[boff + (size_t)o];
                    if (l < L - 1) {
                        if (acc < 0.0) acc = 0.0;
                        if (bf16) acc = round_bf16(acc);
                    }
                    y[o] = acc;
                }
                for (int o = 0; o < nout; ++o) h[o] = y[o];
                woff += (size_t)nout * (size_t)nin;
                boff += (size_t)nout;
            }
            double lp = 0.0;
            for (int blk = 0; 4 * blk < A; ++blk) {
                double z[4];
                or_normals(seed, (uint32_t)e, env_n[e], (uint32_t)blk, OR_TAG_ACTION, z);
                for (int q = 0; q < 4 && 4 * blk + q < A; ++q) {
                    int a = 4 * blk + q;
                    double ls = (double)log_std[a];
                    double mu = h[a];
                    mean[e * (int64_t)A + a] = (float)mu;
                    action[e * (int64_t)A + a] = (float)(mu + exp(ls) * z[q]);
                    lp -= 0.5 * z[q] * z[q] + ls + half_log_2pi;
                }
            }
            if (logp) logp[e] = (float)lp;
        }
        free(h);
        free(y);
    }
}

/* Number of OpenMP threads the batch functions use (for timing reports). */
#ifdef _OPENMP
#include <omp.h>
int or_num_threads(void) { return omp_get_max_threads(); }
#else
int or_num_threads(void) { return 1; }
#endif
