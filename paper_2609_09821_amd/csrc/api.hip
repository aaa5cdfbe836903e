// api.hip -- the C ABI: validation, table preparation and kernel dispatch.
//
// Creation may allocate and synchronise; the hot calls only validate their
// arguments on the host and enqueue kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/instantmimic.h"
#include "launch.h"

using namespace im;

// Parked frames of nested branch points live in LDS (20 floats per slot and
// thread in the stand-in, 256 threads per block): 3 slots keep a block within
// 64 KB.  Humanoid trees need 2.
#define IM_MAX_BRANCH_NESTING 3

struct im_ctx {
    int device = -1;
    int B = 0, D = 0, A = 0, n_clips = 0, L = 0, dtype = 0, n_slots = 0, max_depth = 0;
    int half_slots = 0;   // parked-frame slots of the fused step's half walks
    int64_t max_envs = 0;
    im_config cfg{};
    SkelTab *d_skel = nullptr;
    ClipTab *d_clips = nullptr;
    float4 *d_seg = nullptr;
    std::vector<int> dims, M_pad, K_pad;
    std::vector<void *> d_w;
    std::vector<float *> d_b;
    float *d_log_std = nullptr;
    void *d_ws[2] = {nullptr, nullptr};
    void *d_obs16 = nullptr;   // bf16 [max_envs][K_pad[0]] staging of the observation
    size_t ws_bytes[2] = {0, 0};
    int n_cu = 0;              // compute units of the context's device
    int64_t device_bytes = 0;
    // value head (im_set_critic): hidden layers packed like the policy's,
    // the last layer as an fp32 vector
    struct {
        int L = 0;   // 0: no critic
        std::vector<int> dims, M_pad, K_pad;
        std::vector<void *> d_w;
        std::vector<float *> d_b;
        float *d_head = nullptr;   // [K_head] last-layer weights, zero-padded
        float head_bias = 0.0f;
        int K_head = 0;            // D for a one-layer critic, else M_pad[L-2]
        int64_t bytes = 0;         // device memory of the above
    } critic;
    double *d_partial = nullptr;   // per-block summary sums, [ceil(max_envs/256)][fields]
};

namespace {

thread_local std::string g_err;

im_status fail(im_status s, const std::string &msg)
{
    g_err = msg;
    return s;
}

im_status hip_fail(hipError_t e, const char *what)
{
    return fail(IM_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

bool finite_f(float x) { return std::isfinite(x); }

bool unit_quat(const float *q, double tol)
{
    const double n = std::sqrt((double)q[0] * q[0] + (double)q[1] * q[1] + (double)q[2] * q[2] +
                               (double)q[3] * q[3]);
    return std::isfinite(n) && std::fabs(n - 1.0) <= tol;
}

void free_critic(im_ctx *c)
{
    auto &k = c->critic;
    for (void *p : k.d_w) hipFree(p);
    for (float *p : k.d_b) hipFree(p);
    hipFree(k.d_head);
    k.d_w.clear();
    k.d_b.clear();
    k.d_head = nullptr;
    k.L = 0;
    c->device_bytes -= k.bytes;
    k.bytes = 0;
}

void free_ctx(im_ctx *c)
{
    if (!c) return;
    free_critic(c);
    hipFree(c->d_partial);
    hipFree(c->d_skel);
    hipFree(c->d_clips);
    hipFree(c->d_seg);
    for (void *p : c->d_w) hipFree(p);
    for (float *p : c->d_b) hipFree(p);
    hipFree(c->d_log_std);
    hipFree(c->d_ws[0]);
    hipFree(c->d_ws[1]);
    hipFree(c->d_obs16);
    delete c;
}

template <class T>
hipError_t dev_alloc(im_ctx *c, T **p, size_t bytes)
{
    hipError_t e = hipMalloc((void **)p, bytes);
    if (e == hipSuccess) c->device_bytes += (int64_t)bytes;
    return e;
}

// Preorder tables of the skeleton (host).  Returns an error message or "".
std::string build_skeleton(const im_skeleton *sk, SkelTab *t, int *max_depth)
{
    const int B = sk->n_bodies;
    std::memset(t, 0, sizeof(*t));
    std::vector<std::vector<int>> ch(B);
    for (int b = 1; b < B; ++b) ch[sk->parent[b]].push_back(b);
    std::vector<int> order, depth(B, 0);
    std::vector<int> st{0};
    while (!st.empty()) {
        const int b = st.back();
        st.pop_back();
        order.push_back(b);
        for (auto it = ch[b].rbegin(); it != ch[b].rend(); ++it) {
            depth[*it] = depth[b] + 1;
            st.push_back(*it);
        }
    }
    // nesting level of branch points = number of branch-point proper ancestors
    std::vector<int> nest(B, 0), slot(B, -1);
    int n_slots = 0;
    for (int b = 1; b < B; ++b) {
        const int p = sk->parent[b];
        nest[b] = nest[p] + (ch[p].size() >= 2 ? 1 : 0);
    }
    for (int b = 0; b < B; ++b)
        if (ch[b].size() >= 2) {
            slot[b] = nest[b];
            n_slots = std::max(n_slots, nest[b] + 1);
        }
    // rotational DoFs in body index order (stand-in noise indices)
    std::vector<int> zrot(B, -1);
    int z = 3;
    for (int b = 1; b < B; ++b) {
        if (sk->jtype[b] == IM_JOINT_SPHERICAL) {
            zrot[b] = z;
            z += 3;
        } else if (sk->jtype[b] == IM_JOINT_REVOLUTE) {
            zrot[b] = z;
            z += 1;
        }
    }
    double msum = 0.0;
    for (int b = 0; b < B; ++b) msum += (double)sk->mass[b];
    t->B = B;
    t->n_slots = n_slots;
    t->n_dof = z - 3;
    *max_depth = 0;
    for (int i = 0; i < B; ++i) {
        const int b = order[i];
        t->body[i] = b;
        t->depth[i] = depth[b];
        *max_depth = std::max(*max_depth, depth[b]);
        t->bslot[i] = slot[b];
        t->pslot[i] = -1;
        if (i > 0 && sk->parent[b] != order[i - 1]) {
            const int p = sk->parent[b];
            if (slot[p] < 0) return "internal: preorder parent is not a branch point";
            t->pslot[i] = slot[p];
        }
        t->jtype[i] = sk->jtype[b];
        t->leaf[i] = ch[b].empty() ? 1 : 0;
        t->zrot[i] = zrot[b];
        for (int c = 0; c < 3; ++c) {
            t->offset[i][c] = sk->offset[3 * b + c];
            t->axis[i][c] = sk->axis[3 * b + c];
        }
        t->massw[i] = (float)((double)sk->mass[b] / msum);
    }
    for (int b = 0; b < B; ++b) t->pbody[b] = b > 0 ? sk->parent[b] : -1;
    // future-frame slots: the root, then the leaves in body order
    t->n_ee = 0;
    std::vector<int> slot_of(B, -1);
    for (int b = 1; b < B; ++b)
        if (ch[b].empty()) slot_of[b] = 1 + t->n_ee++;
    slot_of[0] = 0;
    for (int i = 0; i < B; ++i) t->ee_slot[i] = slot_of[order[i]];

    // Two half walks for the fused step.  Half 1 owns the subtrees of a set S
    // of children of one branch point v, half 0 everything else (root
    // included); each walks its bodies plus their ancestors.  Walk lengths:
    // B - |H1| and |H1| + depth(v) + 1; (v, S) minimises the longer one, then
    // their sum.
    std::vector<int> size(B, 1);
    for (int b = B - 1; b > 0; --b) size[sk->parent[b]] += size[b];
    int best_v = -1, best_mask = 0, best_max = B + 1, best_sum = 2 * B + 2;
    for (int v = 0; v < B; ++v) {
        const int nc = (int)ch[v].size();
        if (nc < 2 || nc > 16) continue;
        for (int mask = 1; mask < (1 << nc) - 1; ++mask) {
            int h1 = 0;
            for (int c = 0; c < nc; ++c)
                if (mask >> c & 1) h1 += size[ch[v][c]];
            const int c0 = B - h1, c1 = h1 + depth[v] + 1;
            const int mx = std::max(c0, c1), sm = c0 + c1;
            if (mx < best_max || (mx == best_max && sm < best_sum)) {
                best_v = v;
                best_mask = mask;
                best_max = mx;
                best_sum = sm;
            }
        }
    }
    std::vector<int> owner(B, 0);
    if (best_v >= 0) {
        std::vector<int> stk;
        for (int c = 0; c < (int)ch[best_v].size(); ++c)
            if (best_mask >> c & 1) stk.push_back(ch[best_v][c]);
        while (!stk.empty()) {
            const int b = stk.back();
            stk.pop_back();
            owner[b] = 1;
            for (int cc : ch[b]) stk.push_back(cc);
        }
    }
    std::vector<int> pos_of(B, 0);
    for (int i = 0; i < B; ++i) pos_of[order[i]] = i;
    t->half_slots = 0;
    for (int h = 0; h < 2; ++h) {
        // walk set: owned bodies and their ancestors (closed under parent)
        std::vector<int> in(B, 0);
        for (int b = 0; b < B; ++b)
            if (owner[b] == h)
                for (int x = b; x >= 0 && !in[x]; x = x > 0 ? sk->parent[x] : -1) in[x] = 1;
        in[0] = 1;
        std::vector<std::vector<int>> chw(B);
        for (int b = 1; b < B; ++b)
            if (in[b]) chw[sk->parent[b]].push_back(b);
        std::vector<int> nestw(B, 0), slotw(B, -1), ordw;
        for (int i = 0; i < B; ++i) {            // full preorder restricted to the walk set
            const int b = order[i];
            if (!in[b]) continue;
            ordw.push_back(b);
            if (b > 0) {
                const int p = sk->parent[b];
                nestw[b] = nestw[p] + (chw[p].size() >= 2 ? 1 : 0);
            }
        }
        int ns = 0;
        for (int b : ordw)
            if (chw[b].size() >= 2) {
                slotw[b] = nestw[b];
                ns = std::max(ns, nestw[b] + 1);
            }
        t->half_slots = std::max(t->half_slots, ns);
        auto &w = t->half[h];
        w.n = (int)ordw.size();
        for (int i = 0; i < w.n; ++i) {
            const int b = ordw[i];
            w.body[i] = b;
            w.rec[i] = pos_of[b];
            w.own[i] = owner[b] == h ? 1 : 0;
            w.bslot[i] = slotw[b];
            w.pslot[i] = -1;
            if (i > 0 && sk->parent[b] != ordw[i - 1]) {
                const int p = sk->parent[b];
                if (slotw[p] < 0) return "internal: half-walk parent is not a branch point";
                w.pslot[i] = slotw[p];
            }
            w.jtype[i] = sk->jtype[b];
            w.leaf[i] = ch[b].empty() ? 1 : 0;
            for (int c = 0; c < 3; ++c) w.offset[i][c] = sk->offset[3 * b + c];
            w.offset[i][3] = 0.0f;
            w.massw[i] = (float)((double)sk->mass[b] / msum);
        }
    }
    return "";
}

// Observation width: 15 rows per body, the phase, 9 per future frame of the
// root and each end effector, the previous action.
int64_t obs_width(int B, int n_ee, const im_config *cfg, int A)
{
    return 15 * (int64_t)B + 1 + 9 * (int64_t)cfg->obs_future * (1 + n_ee) +
           (cfg->obs_prev_action ? A : 0);
}

std::string validate(const im_config *cfg, const im_skeleton *sk, const im_clip *clips,
                     int32_t n_clips, const im_policy *pol, int64_t max_envs, im_status *code)
{
    *code = IM_ERR_INVALID_ARG;
    if (!cfg || !sk || !clips || !pol) return "NULL description pointer";
    if (!(cfg->dt > 0.0) || !std::isfinite(cfg->dt)) return "dt must be positive and finite";
    if (!finite_f(cfg->h_term) || !finite_f(cfg->r_min)) return "thresholds must be finite";
    if (cfg->grace < 0) return "grace must be >= 0";
    const float wts[7] = {cfg->c_pose, cfg->w_pos, cfg->w_ee, cfg->c_vel,
                          cfg->w_vel,  cfg->c_com, cfg->w_com};
    for (float w : wts)
        if (!finite_f(w)) return "reward weights must be finite";
    const int B = sk->n_bodies;
    if (B < 1) return "n_bodies must be >= 1";
    if (B > IM_MAX_BODIES) {
        *code = IM_ERR_UNSUPPORTED;
        return "more than IM_MAX_BODIES bodies";
    }
    if (!sk->parent || !sk->jtype || !sk->axis || !sk->offset || !sk->mass)
        return "NULL skeleton array";
    if (sk->parent[0] != -1) return "parent[0] must be -1";
    if (sk->jtype[0] != IM_JOINT_FREE) return "body 0 must have a free joint";
    for (int b = 0; b < B; ++b) {
        if (b > 0 && (sk->parent[b] < 0 || sk->parent[b] >= b))
            return "parent[b] must satisfy 0 <= parent[b] < b (body " + std::to_string(b) + ")";
        if (b > 0 && sk->jtype[b] != IM_JOINT_SPHERICAL && sk->jtype[b] != IM_JOINT_REVOLUTE &&
            sk->jtype[b] != IM_JOINT_FIXED)
            return "invalid joint type at body " + std::to_string(b);
        if (!(sk->mass[b] > 0.0f) || !finite_f(sk->mass[b])) return "masses must be positive";
        for (int c = 0; c < 3; ++c)
            if (!finite_f(sk->offset[3 * b + c]) || !finite_f(sk->axis[3 * b + c]))
                return "offsets/axes must be finite";
        if (b > 0 && sk->jtype[b] == IM_JOINT_REVOLUTE) {
            const float *a = sk->axis + 3 * b;
            const double n = std::sqrt((double)a[0] * a[0] + (double)a[1] * a[1] + (double)a[2] * a[2]);
            if (std::fabs(n - 1.0) > 1e-3) return "revolute axis must be unit";
        }
    }
    if (n_clips < 1) return "n_clips must be >= 1";
    for (int k = 0; k < n_clips; ++k) {
        const im_clip &c = clips[k];
        if (c.n_frames < 2) return "clip " + std::to_string(k) + ": n_frames must be >= 2";
        if (!(c.fps > 0.0f) || !finite_f(c.fps)) return "clip fps must be positive";
        if (!c.root_pos || !c.root_quat || (B > 1 && !c.local_quat)) return "NULL clip array";
        for (int f = 0; f < c.n_frames; ++f) {
            for (int i = 0; i < 3; ++i)
                if (!finite_f(c.root_pos[3 * f + i])) return "clip root positions must be finite";
            if (!unit_quat(c.root_quat + 4 * f, 1e-3)) return "clip root quaternion not unit";
            for (int b = 1; b < B; ++b) {
                const float *q = c.local_quat + 4 * ((int64_t)f * (B - 1) + (b - 1));
                if (sk->jtype[b] == IM_JOINT_FIXED) {
                    if (std::fabs(std::fabs(q[0]) - 1.0f) > 1e-3f || std::fabs(q[1]) > 1e-3f ||
                        std::fabs(q[2]) > 1e-3f || std::fabs(q[3]) > 1e-3f)
                        return "fixed joint with a non-identity clip rotation";
                } else if (!unit_quat(q, 1e-3)) {
                    return "clip joint quaternion not unit (clip " + std::to_string(k) + ")";
                }
            }
        }
    }
    const int L = pol->n_layers;
    if (L < 1 || !pol->dims || !pol->weight || !pol->bias || !pol->log_std)
        return "policy description incomplete";
    if (pol->dtype != IM_DTYPE_F32 && pol->dtype != IM_DTYPE_BF16) return "invalid policy dtype";
    if (cfg->reward_form != IM_REWARD_GROUPED && cfg->reward_form != IM_REWARD_MULTIPLICATIVE)
        return "invalid reward_form";
    const float mw[5] = {cfg->m_jrot, cfg->m_jvel, cfg->m_com, cfg->m_eepos, cfg->m_eerot};
    for (float w : mw)
        if (!finite_f(w)) return "multiplicative reward weights must be finite";
    if (cfg->obs_future < 0 || cfg->obs_future > 4) return "obs_future must be in [0, 4]";
    if (cfg->obs_prev_action != 0 && cfg->obs_prev_action != 1) return "obs_prev_action must be 0 or 1";
    if (cfg->obs_future > 0 && B == 1) {
        *code = IM_ERR_UNSUPPORTED;
        return "future reference frames need at least two bodies";
    }
    {
        std::vector<int> nch(B, 0);
        for (int b = 1; b < B; ++b) nch[sk->parent[b]]++;
        int n_ee = 0;
        for (int b = 0; b < B; ++b) n_ee += nch[b] == 0 ? 1 : 0;
        const int64_t D = obs_width(B, n_ee, cfg, pol->dims[L]);
        if (pol->dims[0] != D)
            return "policy input width must be the observation width " + std::to_string(D);
    }
    for (int l = 0; l <= L; ++l)
        if (pol->dims[l] < 1 || pol->dims[l] > 16384) return "layer widths must be in [1, 16384]";
    if (pol->dims[L] > 128) {
        *code = IM_ERR_UNSUPPORTED;
        return "action width above 128";
    }
    for (int l = 0; l < L; ++l)
        if (!pol->weight[l] || !pol->bias[l]) return "NULL weight or bias";
    for (int a = 0; a < pol->dims[L]; ++a)
        if (!finite_f(pol->log_std[a])) return "log_std must be finite";
    if (max_envs < 1 || max_envs > (int64_t)0xFFFFFFFF) return "max_envs must be in [1, 2^32)";
    *code = IM_OK;
    return "";
}

im_status check_device(const im_ctx *c)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != c->device) return fail(IM_ERR_INVALID_ARG, "call made on another device than the context's");
    return IM_OK;
}

im_status check_env_bufs(const im_ctx *c, const im_env_bufs *b, bool need_outputs)
{
    if (!b) return fail(IM_ERR_INVALID_ARG, "NULL buffers");
    if (b->n_envs < 0 || b->n_envs > (int64_t)0xFFFFFFFF) return fail(IM_ERR_INVALID_ARG, "bad n_envs");
    if (b->ld < b->n_envs || b->ld < 1) return fail(IM_ERR_INVALID_ARG, "ld must be >= n_envs and >= 1");
    if (!b->body_pos || !b->body_quat || !b->body_linvel || !b->body_angvel || !b->env_clip ||
        !b->env_phase || !b->env_t || !b->env_n || !b->obs)
        return fail(IM_ERR_INVALID_ARG, "NULL env buffer");
    if (need_outputs && (!b->reward || !b->terminated || !b->truncated))
        return fail(IM_ERR_INVALID_ARG, "NULL output buffer");
    if (need_outputs && c->cfg.obs_prev_action && !b->prev_action)
        return fail(IM_ERR_INVALID_ARG, "the observation needs prev_action");
    return IM_OK;
}

EnvArgs env_args(const im_ctx *c, const im_env_bufs *b)
{
    EnvArgs a{};
    a.sk = c->d_skel;
    a.clips = c->d_clips;
    a.seg = c->d_seg;
    a.pos = b->body_pos;
    a.quat = b->body_quat;
    a.linvel = b->body_linvel;
    a.angvel = b->body_angvel;
    a.env_clip = b->env_clip;
    a.env_phase = b->env_phase;
    a.env_t = b->env_t;
    a.env_n = b->env_n;
    a.reward = b->reward;
    a.term = b->terminated;
    a.trunc = b->truncated;
    a.obs = b->obs;
    a.ref_frame = b->ref_frame;
    a.mask = nullptr;
    a.n = b->n_envs;
    a.ld = b->ld;
    a.seed = c->cfg.seed;
    a.n_clips = c->n_clips;
    a.grace = c->cfg.grace;
    a.h_term = c->cfg.h_term;
    a.r_min = c->cfg.r_min;
    a.c_pose = c->cfg.c_pose;
    a.w_pos = c->cfg.w_pos;
    a.w_ee = c->cfg.w_ee;
    a.c_vel = c->cfg.c_vel;
    a.w_vel = c->cfg.w_vel;
    a.c_com = c->cfg.c_com;
    a.w_com = c->cfg.w_com;
    a.reward_form = c->cfg.reward_form;
    a.obs_prev = c->cfg.obs_prev_action;
    a.m_jrot = c->cfg.m_jrot;
    a.m_jvel = c->cfg.m_jvel;
    a.m_com = c->cfg.m_com;
    a.m_eepos = c->cfg.m_eepos;
    a.m_eerot = c->cfg.m_eerot;
    a.obs_future = c->cfg.obs_future;
    a.obs_base = 15 * c->B + 1;
    a.A = c->A;
    a.prev_action = c->cfg.obs_prev_action ? b->prev_action : nullptr;
    return a;
}

}  // namespace

extern "C" {

const char *im_status_str(im_status s)
{
    switch (s) {
        case IM_OK: return "IM_OK";
        case IM_ERR_INVALID_ARG: return "IM_ERR_INVALID_ARG";
        case IM_ERR_UNSUPPORTED: return "IM_ERR_UNSUPPORTED";
        case IM_ERR_OOM: return "IM_ERR_OOM";
        case IM_ERR_HIP: return "IM_ERR_HIP";
    }
    return "unknown im_status";
}

const char *im_last_error(void) { return g_err.c_str(); }

im_status im_create(const im_config *cfg, const im_skeleton *sk, const im_clip *clips,
                    int32_t n_clips, const im_policy *pol, int64_t max_envs, im_ctx **out)
{
    if (!out) return fail(IM_ERR_INVALID_ARG, "NULL out pointer");
    *out = nullptr;
    im_status code;
    std::string msg = validate(cfg, sk, clips, n_clips, pol, max_envs, &code);
    if (code != IM_OK) return fail(code, msg);

    SkelTab tab;
    int max_depth = 0;
    msg = build_skeleton(sk, &tab, &max_depth);
    if (!msg.empty()) return fail(IM_ERR_INVALID_ARG, msg);
    if (tab.n_slots > IM_MAX_BRANCH_NESTING || tab.half_slots > IM_MAX_BRANCH_NESTING)
        return fail(IM_ERR_UNSUPPORTED, "branch points nested deeper than " +
                                            std::to_string(IM_MAX_BRANCH_NESTING));

    im_ctx *c = new im_ctx();
    hipError_t e = hipGetDevice(&c->device);
    if (e != hipSuccess) {
        free_ctx(c);
        return hip_fail(e, "hipGetDevice");
    }
    if (hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device) != hipSuccess)
        c->n_cu = 0;
    c->B = sk->n_bodies;
    c->D = (int)obs_width(c->B, tab.n_ee, cfg, pol->dims[pol->n_layers]);
    c->L = pol->n_layers;
    c->A = pol->dims[c->L];
    c->n_clips = n_clips;
    c->dtype = pol->dtype;
    c->n_slots = tab.n_slots;
    c->half_slots = tab.half_slots;
    c->max_depth = max_depth;
    c->max_envs = max_envs;
    c->cfg = *cfg;

#define IM_TRY_ALLOC(ptr, bytes)                                                              \
    do {                                                                                      \
        if (dev_alloc(c, &(ptr), (bytes)) != hipSuccess) {                                    \
            free_ctx(c);                                                                      \
            return fail(IM_ERR_OOM, "device allocation failed (" + std::to_string(bytes) +    \
                                        " bytes)");                                           \
        }                                                                                     \
    } while (0)
#define IM_TRY_HIP(call, what)                                                                \
    do {                                                                                      \
        hipError_t e_ = (call);                                                               \
        if (e_ != hipSuccess) {                                                               \
            im_status s_ = hip_fail(e_, what);                                                \
            free_ctx(c);                                                                      \
            return s_;                                                                        \
        }                                                                                     \
    } while (0)

    // skeleton and per-clip tables
    IM_TRY_ALLOC(c->d_skel, sizeof(SkelTab));
    IM_TRY_HIP(hipMemcpy(c->d_skel, &tab, sizeof(SkelTab), hipMemcpyHostToDevice), "upload skeleton");
    std::vector<ClipTab> ct(n_clips);
    int64_t seg_total = 0;
    const int stride = seg_stride(c->B);
    for (int k = 0; k < n_clips; ++k) {
        const int F = clips[k].n_frames;
        ct[k].F = F;
        ct[k].dphi = (float)(cfg->dt * (double)clips[k].fps / (double)(F - 1));
        ct[k].fm1 = (float)(F - 1);
        if (seg_total > (int64_t)0x7FFFFFFF) {
            free_ctx(c);
            return fail(IM_ERR_UNSUPPORTED, "segment table too large");
        }
        ct[k].seg_base = (int32_t)seg_total;
        seg_total += (int64_t)(F - 1) * stride;
    }
    IM_TRY_ALLOC(c->d_clips, sizeof(ClipTab) * n_clips);
    IM_TRY_HIP(hipMemcpy(c->d_clips, ct.data(), sizeof(ClipTab) * n_clips, hipMemcpyHostToDevice),
               "upload clip table");
    IM_TRY_ALLOC(c->d_seg, sizeof(float4) * seg_total);

    // reference segments: upload each clip's frames and pack them on the device
    for (int k = 0; k < n_clips; ++k) {
        const int F = clips[k].n_frames;
        const size_t nrp = 3 * (size_t)F, nrq = 4 * (size_t)F,
                     nlq = 4 * (size_t)F * (size_t)std::max(c->B - 1, 1);
        float *tmp = nullptr;
        if (hipMalloc((void **)&tmp, sizeof(float) * (nrp + nrq + nlq)) != hipSuccess) {
            free_ctx(c);
            return fail(IM_ERR_OOM, "device allocation failed (clip staging)");
        }
        hipError_t err = hipMemcpy(tmp, clips[k].root_pos, sizeof(float) * nrp, hipMemcpyHostToDevice);
        if (err == hipSuccess)
            err = hipMemcpy(tmp + nrp, clips[k].root_quat, sizeof(float) * nrq, hipMemcpyHostToDevice);
        if (err == hipSuccess && c->B > 1)
            err = hipMemcpy(tmp + nrp + nrq, clips[k].local_quat,
                            sizeof(float) * 4 * (size_t)F * (size_t)(c->B - 1), hipMemcpyHostToDevice);
        if (err == hipSuccess)
            err = launch_pack_segments(c->d_skel, F, (double)clips[k].fps, tmp, tmp + nrp,
                                       tmp + nrp + nrq, c->d_seg + ct[k].seg_base, nullptr);
        if (err == hipSuccess) err = hipDeviceSynchronize();
        hipFree(tmp);
        if (err != hipSuccess) {
            free_ctx(c);
            return hip_fail(err, "pack reference segments");
        }
    }

    // policy: zero-padded weight layout [M_pad][K_pad], biases [M_pad]
    const size_t esz = pol->dtype == IM_DTYPE_BF16 ? 2 : 4;
    c->dims.assign(pol->dims, pol->dims + c->L + 1);
    c->M_pad.resize(c->L);
    c->K_pad.resize(c->L);
    int64_t ws_width = 0;
    for (int l = 0; l < c->L; ++l) {
        const bool last = l == c->L - 1;
        // hidden widths padded to the 256-feature macro tile, the action width
        // to one MFMA tile row (32); K to the 64-element GEMM step
        c->M_pad[l] = (int)round_up(c->dims[l + 1], last ? 32 : 256);
        c->K_pad[l] = l == 0 ? (int)round_up(c->dims[0], 64) : c->M_pad[l - 1];
        if (!last) ws_width = std::max<int64_t>(ws_width, c->M_pad[l]);
        const int M = c->dims[l + 1], K = c->dims[l];
        std::vector<uint8_t> wbuf((size_t)c->M_pad[l] * c->K_pad[l] * esz, 0);
        for (int m = 0; m < M; ++m)
            std::memcpy(wbuf.data() + ((size_t)m * c->K_pad[l]) * esz,
                        (const uint8_t *)pol->weight[l] + (size_t)m * K * esz, (size_t)K * esz);
        std::vector<float> bbuf(c->M_pad[l], 0.0f);
        std::memcpy(bbuf.data(), pol->bias[l], sizeof(float) * M);
        void *dw = nullptr;
        float *db = nullptr;
        IM_TRY_ALLOC(dw, wbuf.size());
        c->d_w.push_back(dw);
        IM_TRY_ALLOC(db, sizeof(float) * bbuf.size());
        c->d_b.push_back(db);
        IM_TRY_HIP(hipMemcpy(dw, wbuf.data(), wbuf.size(), hipMemcpyHostToDevice), "upload weights");
        IM_TRY_HIP(hipMemcpy(db, bbuf.data(), sizeof(float) * bbuf.size(), hipMemcpyHostToDevice),
                   "upload biases");
    }
    IM_TRY_ALLOC(c->d_log_std, sizeof(float) * c->A);
    IM_TRY_HIP(hipMemcpy(c->d_log_std, pol->log_std, sizeof(float) * c->A, hipMemcpyHostToDevice),
               "upload log_std");
    IM_TRY_ALLOC(c->d_partial,
                  sizeof(double) * IM_SUMMARY_FIELDS * (size_t)((max_envs + 255) / 256));
    if (c->L >= 2) {
        const size_t wsb = (size_t)max_envs * (size_t)ws_width * esz;
        IM_TRY_ALLOC(c->d_ws[0], wsb);
        c->ws_bytes[0] = wsb;
        if (c->L >= 3) {
            IM_TRY_ALLOC(c->d_ws[1], wsb);
            c->ws_bytes[1] = wsb;
        }
        // large bf16 batches stage the observation as bf16 rows for the first layer
        if (pol->dtype == IM_DTYPE_BF16 && max_envs > SMALL_BATCH)
            IM_TRY_ALLOC(c->d_obs16, (size_t)max_envs * (size_t)c->K_pad[0] * 2);
    }
#undef IM_TRY_ALLOC
#undef IM_TRY_HIP
    *out = c;
    return IM_OK;
}

im_status im_destroy(im_ctx *ctx)
{
    if (!ctx) return fail(IM_ERR_INVALID_ARG, "NULL context");
    free_ctx(ctx);
    return IM_OK;
}

im_status im_get_info(const im_ctx *c, im_info *info)
{
    if (!c || !info) return fail(IM_ERR_INVALID_ARG, "NULL argument");
    info->n_bodies = c->B;
    info->obs_dim = c->D;
    info->action_dim = c->A;
    info->n_clips = c->n_clips;
    info->n_layers = c->L;
    info->policy_dtype = c->dtype;
    info->max_depth = c->max_depth;
    info->max_envs = c->max_envs;
    info->device_bytes = c->device_bytes;
    return IM_OK;
}

im_status im_env_step_fused(im_ctx *c, const im_env_bufs *b, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    im_status s = check_env_bufs(c, b, true);
    if (s != IM_OK) return s;
    if ((s = check_device(c)) != IM_OK) return s;
    const EnvArgs a = env_args(c, b);
    hipError_t e = launch_env_step(c->n_slots, c->half_slots, a, (hipStream_t)stream);
    return e == hipSuccess ? IM_OK : hip_fail(e, "env_step launch");
}

im_status im_reset_envs(im_ctx *c, const im_env_bufs *b, const uint8_t *mask, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    im_status s = check_env_bufs(c, b, false);
    if (s != IM_OK) return s;
    if ((s = check_device(c)) != IM_OK) return s;
    EnvArgs a = env_args(c, b);
    a.mask = mask;
    hipError_t e = launch_reset(c->n_slots, a, (hipStream_t)stream);
    return e == hipSuccess ? IM_OK : hip_fail(e, "reset launch");
}

im_status im_standin_physics(im_ctx *c, const im_env_bufs *b, float sigma_joint, float sigma_vel,
                             void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    im_status s = check_env_bufs(c, b, false);
    if (s != IM_OK) return s;
    if (!finite_f(sigma_joint) || !finite_f(sigma_vel) || sigma_joint < 0.0f || sigma_vel < 0.0f)
        return fail(IM_ERR_INVALID_ARG, "sigmas must be finite and >= 0");
    if ((s = check_device(c)) != IM_OK) return s;
    EnvArgs a = env_args(c, b);
    a.sigma_joint = sigma_joint;
    a.sigma_vel = sigma_vel;
    hipError_t e = launch_standin(c->n_slots, a, (hipStream_t)stream);
    return e == hipSuccess ? IM_OK : hip_fail(e, "stand-in launch");
}

im_status im_policy_act(im_ctx *c, const float *obs, int64_t ld_obs, const uint32_t *env_n,
                        int64_t n_envs, float *mean, float *action, float *logp, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    if (!obs || !env_n || !mean || !action) return fail(IM_ERR_INVALID_ARG, "NULL buffer");
    if (n_envs < 0 || n_envs > c->max_envs) return fail(IM_ERR_INVALID_ARG, "n_envs must be in [0, max_envs]");
    if (ld_obs < n_envs || ld_obs < 1) return fail(IM_ERR_INVALID_ARG, "ld_obs must be >= n_envs");
    im_status s = check_device(c);
    if (s != IM_OK) return s;
    const bool bf16 = c->dtype == IM_DTYPE_BF16;
    const uint64_t esz = bf16 ? 2 : 4;
    // buffer loads address with 32-bit byte offsets
    for (int l = 0; l < c->L; ++l) {
        const uint64_t xb = l == 0 ? (uint64_t)c->D * (uint64_t)ld_obs * 4
                                   : (uint64_t)n_envs * (uint64_t)c->M_pad[l - 1] * esz;
        if (xb > 0xFFFFFFF0ull)
            return fail(IM_ERR_UNSUPPORTED, "policy input of layer " + std::to_string(l) +
                                                " exceeds 4 GiB");
    }
    if (c->d_obs16 && (uint64_t)n_envs * (uint64_t)c->K_pad[0] * 2 > 0xFFFFFFF0ull)
        return fail(IM_ERR_UNSUPPORTED, "staged policy input exceeds 4 GiB");
    for (int l = 0; l < c->L; ++l) {
        GemmArgs g{};
        const bool last = l == c->L - 1;
        g.x = l == 0 ? (const void *)obs : c->d_ws[(l - 1) & 1];
        g.ld_x = l == 0 ? ld_obs : c->M_pad[l - 1];
        g.x_bytes = (uint32_t)(l == 0 ? (uint64_t)c->D * (uint64_t)ld_obs * 4
                                      : (uint64_t)n_envs * (uint64_t)c->M_pad[l - 1] * esz);
        g.w_bytes = (uint32_t)((uint64_t)c->M_pad[l] * (uint64_t)c->K_pad[l] * esz);
        g.w = c->d_w[l];
        g.bias = c->d_b[l];
        g.K_pad = c->K_pad[l];
        g.K_valid = l == 0 ? c->D : c->K_pad[l];
        g.N = n_envs;
        g.x16 = l == 0 ? c->d_obs16 : nullptr;
        g.n_cu = c->n_cu;
        if (!last) {
            g.y = c->d_ws[l & 1];
            g.ld_y = c->M_pad[l];
        } else {
            g.mean = mean;
            g.action = action;
            g.logp = logp;
            g.env_n = env_n;
            g.log_std = c->d_log_std;
            g.A = c->A;
            g.seed = c->cfg.seed;
        }
        hipError_t e = launch_policy_layer(bf16, l == 0, last, g, c->M_pad[l], (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "policy layer launch");
    }
    return IM_OK;
}

}  // extern "C"

namespace {

// Hidden layers 0..n_hidden-1 of a packed MLP (bias, ReLU, the dtype's
// rounding) on the observation; the last activations end in d_ws[(n_hidden-1) & 1].
im_status mlp_hidden(im_ctx *c, int n_hidden, const std::vector<int> &M_pad,
                     const std::vector<int> &K_pad, const std::vector<void *> &d_w,
                     const std::vector<float *> &d_b, const float *obs, int64_t ld_obs,
                     int64_t n_envs, hipStream_t stream)
{
    const bool bf16 = c->dtype == IM_DTYPE_BF16;
    const uint64_t esz = bf16 ? 2 : 4;
    for (int l = 0; l < n_hidden; ++l) {
        GemmArgs g{};
        g.x = l == 0 ? (const void *)obs : c->d_ws[(l - 1) & 1];
        g.ld_x = l == 0 ? ld_obs : M_pad[l - 1];
        g.x_bytes = (uint32_t)(l == 0 ? (uint64_t)c->D * (uint64_t)ld_obs * 4
                                      : (uint64_t)n_envs * (uint64_t)M_pad[l - 1] * esz);
        g.w_bytes = (uint32_t)((uint64_t)M_pad[l] * (uint64_t)K_pad[l] * esz);
        g.w = d_w[l];
        g.bias = d_b[l];
        g.K_pad = K_pad[l];
        g.K_valid = l == 0 ? c->D : K_pad[l];
        g.N = n_envs;
        g.x16 = l == 0 ? c->d_obs16 : nullptr;
        g.n_cu = c->n_cu;
        g.y = c->d_ws[l & 1];
        g.ld_y = M_pad[l];
        hipError_t e = launch_policy_layer(bf16, l == 0, false, g, M_pad[l], stream);
        if (e != hipSuccess) return hip_fail(e, "hidden layer launch");
    }
    return IM_OK;
}

// Grow workspace buffer i to at least `bytes`.
im_status ensure_ws(im_ctx *c, int i, size_t bytes)
{
    if (c->ws_bytes[i] >= bytes) return IM_OK;
    hipFree(c->d_ws[i]);
    c->device_bytes -= (int64_t)c->ws_bytes[i];
    c->d_ws[i] = nullptr;
    c->ws_bytes[i] = 0;
    if (dev_alloc(c, &c->d_ws[i], bytes) != hipSuccess)
        return fail(IM_ERR_OOM, "device allocation failed (workspace)");
    c->ws_bytes[i] = bytes;
    return IM_OK;
}

}  // namespace

extern "C" {

im_status im_set_critic(im_ctx *c, const im_policy *k)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    if (!k) return fail(IM_ERR_INVALID_ARG, "NULL critic");
    const int L = k->n_layers;
    if (L < 1 || !k->dims || !k->weight || !k->bias) return fail(IM_ERR_INVALID_ARG, "critic description incomplete");
    if (k->dtype != c->dtype) return fail(IM_ERR_INVALID_ARG, "critic dtype must be the policy's");
    if (k->dims[0] != c->D)
        return fail(IM_ERR_INVALID_ARG, "critic input width must be the observation width " +
                                            std::to_string(c->D));
    if (k->dims[L] != 1) return fail(IM_ERR_INVALID_ARG, "critic output width must be 1");
    for (int l = 0; l <= L; ++l)
        if (k->dims[l] < 1 || k->dims[l] > 16384)
            return fail(IM_ERR_INVALID_ARG, "layer widths must be in [1, 16384]");
    for (int l = 0; l < L; ++l)
        if (!k->weight[l] || !k->bias[l]) return fail(IM_ERR_INVALID_ARG, "NULL weight or bias");
    im_status s = check_device(c);
    if (s != IM_OK) return s;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "synchronise before replacing the critic");
    free_critic(c);
    auto &cr = c->critic;
    const bool bf16 = c->dtype == IM_DTYPE_BF16;
    const size_t esz = bf16 ? 2 : 4;
    cr.dims.assign(k->dims, k->dims + L + 1);
    cr.M_pad.assign(L - 1, 0);
    cr.K_pad.assign(L - 1, 0);
    int64_t ws_width = 0;
    auto alloc = [&](auto **p, size_t bytes) {
        if (dev_alloc(c, p, bytes) != hipSuccess) return false;
        cr.bytes += (int64_t)bytes;
        return true;
    };
    auto oom = [&](const char *what) {
        free_critic(c);
        return fail(IM_ERR_OOM, std::string("device allocation failed (") + what + ")");
    };
    auto upload_fail = [&](hipError_t err, const char *what) {
        free_critic(c);
        return hip_fail(err, what);
    };
    for (int l = 0; l < L - 1; ++l) {
        cr.M_pad[l] = (int)round_up(cr.dims[l + 1], 256);
        cr.K_pad[l] = l == 0 ? (int)round_up(cr.dims[0], 64) : cr.M_pad[l - 1];
        ws_width = std::max<int64_t>(ws_width, cr.M_pad[l]);
        const int M = cr.dims[l + 1], K = cr.dims[l];
        std::vector<uint8_t> wbuf((size_t)cr.M_pad[l] * cr.K_pad[l] * esz, 0);
        for (int m = 0; m < M; ++m)
            std::memcpy(wbuf.data() + ((size_t)m * cr.K_pad[l]) * esz,
                        (const uint8_t *)k->weight[l] + (size_t)m * K * esz, (size_t)K * esz);
        std::vector<float> bbuf(cr.M_pad[l], 0.0f);
        std::memcpy(bbuf.data(), k->bias[l], sizeof(float) * M);
        void *dw = nullptr;
        float *db = nullptr;
        if (!alloc(&dw, wbuf.size())) return oom("critic weights");
        cr.d_w.push_back(dw);
        if (!alloc(&db, sizeof(float) * bbuf.size())) return oom("critic biases");
        cr.d_b.push_back(db);
        if ((e = hipMemcpy(dw, wbuf.data(), wbuf.size(), hipMemcpyHostToDevice)) != hipSuccess)
            return upload_fail(e, "upload critic weights");
        if ((e = hipMemcpy(db, bbuf.data(), sizeof(float) * bbuf.size(), hipMemcpyHostToDevice)) !=
            hipSuccess)
            return upload_fail(e, "upload critic biases");
    }
    // last layer as an fp32 vector (bf16 weights convert exactly)
    cr.K_head = L == 1 ? c->D : cr.M_pad[L - 2];
    std::vector<float> head(cr.K_head, 0.0f);
    const int K = cr.dims[L - 1];
    for (int i = 0; i < K; ++i) {
        if (bf16) {
            uint16_t h;
            std::memcpy(&h, (const uint8_t *)k->weight[L - 1] + 2 * (size_t)i, 2);
            const uint32_t u = (uint32_t)h << 16;
            std::memcpy(&head[i], &u, 4);
        } else {
            std::memcpy(&head[i], (const uint8_t *)k->weight[L - 1] + 4 * (size_t)i, 4);
        }
    }
    cr.head_bias = k->bias[L - 1][0];
    if (!alloc(&cr.d_head, sizeof(float) * head.size())) return oom("critic head");
    if ((e = hipMemcpy(cr.d_head, head.data(), sizeof(float) * head.size(), hipMemcpyHostToDevice)) !=
        hipSuccess)
        return upload_fail(e, "upload critic head");
    // workspace for the hidden activations and the bf16 observation staging
    if (L >= 2) {
        const size_t wsb = (size_t)c->max_envs * (size_t)ws_width * esz;
        if ((s = ensure_ws(c, 0, wsb)) != IM_OK || (L >= 3 && (s = ensure_ws(c, 1, wsb)) != IM_OK)) {
            free_critic(c);
            return s;
        }
        if (bf16 && c->max_envs > SMALL_BATCH && !c->d_obs16 &&
            dev_alloc(c, &c->d_obs16, (size_t)c->max_envs * (size_t)round_up(c->D, 64) * 2) !=
                hipSuccess)
            return oom("observation staging");
    }
    cr.L = L;
    return IM_OK;
}

im_status im_value(im_ctx *c, const float *obs, int64_t ld_obs, int64_t n_envs, float *value,
                   void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    const auto &cr = c->critic;
    if (cr.L == 0) return fail(IM_ERR_INVALID_ARG, "no critic (im_set_critic)");
    if (!obs || !value) return fail(IM_ERR_INVALID_ARG, "NULL buffer");
    if (n_envs < 0 || n_envs > c->max_envs) return fail(IM_ERR_INVALID_ARG, "n_envs must be in [0, max_envs]");
    if (ld_obs < n_envs || ld_obs < 1) return fail(IM_ERR_INVALID_ARG, "ld_obs must be >= n_envs");
    im_status s = check_device(c);
    if (s != IM_OK) return s;
    const bool bf16 = c->dtype == IM_DTYPE_BF16;
    const uint64_t esz = bf16 ? 2 : 4;
    if ((uint64_t)c->D * (uint64_t)ld_obs * 4 > 0xFFFFFFF0ull)
        return fail(IM_ERR_UNSUPPORTED, "critic input exceeds 4 GiB");
    for (int l = 1; l < cr.L - 1; ++l)
        if ((uint64_t)n_envs * (uint64_t)cr.M_pad[l - 1] * esz > 0xFFFFFFF0ull)
            return fail(IM_ERR_UNSUPPORTED, "critic layer input exceeds 4 GiB");
    if (c->d_obs16 && (uint64_t)n_envs * (uint64_t)round_up(c->D, 64) * 2 > 0xFFFFFFF0ull)
        return fail(IM_ERR_UNSUPPORTED, "staged critic input exceeds 4 GiB");
    const hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if (cr.L == 1) {
        e = launch_value_head_obs(obs, ld_obs, c->D, cr.d_head, cr.head_bias, bf16, n_envs, value, st);
    } else {
        if ((s = mlp_hidden(c, cr.L - 1, cr.M_pad, cr.K_pad, cr.d_w, cr.d_b, obs, ld_obs, n_envs,
                            st)) != IM_OK)
            return s;
        e = launch_value_head_rows(bf16, c->d_ws[(cr.L - 2) & 1], cr.K_head, cr.K_head, cr.d_head,
                                   cr.head_bias, n_envs, value, st);
    }
    return e == hipSuccess ? IM_OK : hip_fail(e, "value head launch");
}

im_status im_gae(im_ctx *c, const im_rollout *r, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    if (!r) return fail(IM_ERR_INVALID_ARG, "NULL rollout");
    if (r->T < 1) return fail(IM_ERR_INVALID_ARG, "T must be >= 1");
    if (r->n_envs < 0 || r->n_envs > c->max_envs)
        return fail(IM_ERR_INVALID_ARG, "n_envs must be in [0, max_envs]");
    if (r->ld < r->n_envs || r->ld < 1) return fail(IM_ERR_INVALID_ARG, "ld must be >= n_envs and >= 1");
    if (!r->reward || !r->terminated || !r->truncated || !r->value || !r->advantage || !r->ret)
        return fail(IM_ERR_INVALID_ARG, "NULL rollout buffer");
    if (r->summary && (!r->ep_return || !r->ep_length))
        return fail(IM_ERR_INVALID_ARG, "summaries need ep_return and ep_length");
    if (!(r->gamma >= 0.0f && r->gamma <= 1.0f) || !(r->lambda >= 0.0f && r->lambda <= 1.0f))
        return fail(IM_ERR_INVALID_ARG, "gamma and lambda must be in [0, 1]");
    im_status s = check_device(c);
    if (s != IM_OK) return s;
    GaeArgs g{};
    g.T = r->T;
    g.n = r->n_envs;
    g.ld = r->ld;
    g.gamma = (double)r->gamma;
    g.lambda = (double)r->lambda;
    g.reward = r->reward;
    g.term = r->terminated;
    g.trunc = r->truncated;
    g.value = r->value;
    g.adv = r->advantage;
    g.ret = r->ret;
    g.ep_return = r->ep_return;
    g.ep_length = r->ep_length;
    g.summary = r->summary;
    g.partial = c->d_partial;
    hipError_t e = launch_gae(g, (hipStream_t)stream);
    return e == hipSuccess ? IM_OK : hip_fail(e, "gae launch");
}

}  // extern "C"
