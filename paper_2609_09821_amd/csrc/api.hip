// api.hip -- the C ABI: validation, table preparation and kernel dispatch.
//
// Creation may allocate and synchronise; the hot calls only validate their
// arguments on the host and enqueue kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/instantmimic.h"
#include "launch.h"

using namespace im;

// Parked frames of nested branch points live in LDS (20 floats per slot and
// thread in the stand-in, 256 threads per block): 3 slots keep a block within
// 64 KB.  Humanoid trees need 2.
#define IM_MAX_BRANCH_NESTING 3

namespace im {
struct TrainState;
void free_train(TrainState *t);
}  // namespace im

struct im_ctx {
    int device = -1;
    int B = 0, D = 0, A = 0, n_clips = 0, L = 0, dtype = 0, n_slots = 0, max_depth = 0;
    int half_slots = 0;   // parked-frame slots of the fused step's half walks
    int n_paths = 0;      // root-to-leaf walks of the path-split fused step (0: none)
    int path_slots = 0;
    int64_t max_envs = 0;
    im_config cfg{};
    SkelTab *d_skel = nullptr;
    ClipTab *d_clips = nullptr;
    float4 *d_seg = nullptr;
    std::vector<int> dims, M_pad, K_pad;
    std::vector<void *> d_w;
    std::vector<float *> d_b;
    // bf16 policies that the one-launch policy kernel holds: each layer's
    // weights again, in MFMA fragment order (empty otherwise)
    std::vector<uint16_t *> d_wf;
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
        std::vector<uint16_t *> d_wf;   // bf16 critics the one-launch kernel holds: the hidden
                                        // layers' weights in MFMA fragment order (else empty)
        float *d_head = nullptr;   // [K_head + 1]: last-layer weights (zero-padded), then its bias
        int K_head = 0;            // D for a one-layer critic, else M_pad[L-2]
        int64_t bytes = 0;         // device memory of the above
    } critic;
    double *d_partial = nullptr;   // per-block summary sums, [ceil(max_envs/256)][fields]
    im::TrainState *train = nullptr;   // PPO update state (im_ppo_setup)
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

// A bf16 policy whose widths the one-launch policy kernel holds.
bool fused_policy_fits(const im_ctx *c)
{
    if (c->L > FUSED_MAX_LAYERS || c->K_pad[0] > FUSED_MAX_WIDTH || c->M_pad[c->L - 1] > 128)
        return false;
    for (int l = 0; l + 1 < c->L; ++l)
        if (c->M_pad[l] > FUSED_MAX_WIDTH) return false;
    return true;
}

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
    for (uint16_t *p : k.d_wf) hipFree(p);
    hipFree(k.d_head);
    k.d_w.clear();
    k.d_b.clear();
    k.d_wf.clear();
    k.d_head = nullptr;
    k.L = 0;
    c->device_bytes -= k.bytes;
    k.bytes = 0;
}

void free_ctx(im_ctx *c)
{
    if (!c) return;
    im::free_train(c->train);
    free_critic(c);
    hipFree(c->d_partial);
    hipFree(c->d_skel);
    hipFree(c->d_clips);
    hipFree(c->d_seg);
    for (void *p : c->d_w) hipFree(p);
    for (float *p : c->d_b) hipFree(p);
    for (uint16_t *p : c->d_wf) hipFree(p);
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
    // The walk of the bodies with own_of[b] == h and their ancestors, in the
    // full preorder; *slots = the parked-frame slots it needs.
    auto build_walk = [&](const std::vector<int> &own_of, int h, SkelTab::PartWalk &w,
                          int *slots) -> std::string {
        std::vector<int> in(B, 0);   // walk set: owned bodies and their ancestors
        for (int b = 0; b < B; ++b)
            if (own_of[b] == h)
                for (int x = b; x >= 0 && !in[x]; x = x > 0 ? sk->parent[x] : -1) in[x] = 1;
        in[0] = 1;
        std::vector<std::vector<int>> chw(B);
        for (int b = 1; b < B; ++b)
            if (in[b]) chw[sk->parent[b]].push_back(b);
        std::vector<int> nestw(B, 0), slotw(B, -1), ordw;
        for (int i = 0; i < B; ++i) {
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
        *slots = ns;
        w.n = (int)ordw.size();
        w.n_own = 0;
        for (int i = 0; i < w.n; ++i) {
            const int b = ordw[i];
            w.body[i] = b;
            w.rec[i] = pos_of[b];
            w.own[i] = own_of[b] == h ? 1 : 0;
            if (w.own[i]) w.own_body[w.n_own++] = b;
            w.bslot[i] = slotw[b];
            w.pslot[i] = -1;
            if (i > 0 && sk->parent[b] != ordw[i - 1]) {
                const int p = sk->parent[b];
                if (slotw[p] < 0) return "internal: part-walk parent is not a branch point";
                w.pslot[i] = slotw[p];
            }
            w.jtype[i] = sk->jtype[b];
            w.leaf[i] = ch[b].empty() ? 1 : 0;
            for (int c = 0; c < 3; ++c) w.offset[i][c] = sk->offset[3 * b + c];
            w.offset[i][3] = 0.0f;
            w.massw[i] = (float)((double)sk->mass[b] / msum);
        }
        return "";
    };
    t->half_slots = 0;
    for (int h = 0; h < 2; ++h) {
        int ns = 0;
        const std::string err = build_walk(owner, h, t->half[h], &ns);
        if (!err.empty()) return err;
        t->half_slots = std::max(t->half_slots, ns);
    }
    // Path walks: one per leaf (preorder), each owning the bodies of its
    // root-to-leaf path not owned by an earlier path.
    std::vector<int> leaves;
    for (int i = 0; i < B; ++i)
        if (ch[order[i]].empty() && order[i] != 0) leaves.push_back(order[i]);
    t->n_paths = 0;
    t->path_slots = 0;
    if (leaves.size() >= 2 && leaves.size() <= (size_t)IM_MAX_PATHS) {
        std::vector<int> own_path(B, -1);
        for (int p = 0; p < (int)leaves.size(); ++p)
            for (int x = leaves[p]; x >= 0; x = x > 0 ? sk->parent[x] : -1)
                if (own_path[x] < 0) own_path[x] = p;
        for (int p = 0; p < (int)leaves.size(); ++p) {
            int ns = 0;
            const std::string err = build_walk(own_path, p, t->path[p], &ns);
            if (!err.empty()) return err;
            t->path_slots = std::max(t->path_slots, ns);
        }
        t->n_paths = (int)leaves.size();
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
    if (cfg->env_split < IM_SPLIT_AUTO || cfg->env_split > IM_SPLIT_PATHS)
        return "env_split must be one of IM_SPLIT_AUTO, IM_SPLIT_ONE, IM_SPLIT_HALVES, IM_SPLIT_PATHS";
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
    if (pol->dims[L] > im::MAX_ACTIONS) {
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
    if (cfg->env_split == IM_SPLIT_PATHS && tab.n_paths < 2)
        return fail(IM_ERR_UNSUPPORTED, "env_split IM_SPLIT_PATHS needs 2.." +
                                            std::to_string(IM_MAX_PATHS) + " leaves");

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
    c->n_paths = tab.n_paths;
    c->path_slots = tab.path_slots;
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
    if (pol->dtype == IM_DTYPE_BF16 && fused_policy_fits(c)) {
        for (int l = 0; l < c->L; ++l) {
            const int M = c->dims[l + 1], K = c->dims[l], nks = c->K_pad[l] / 64;
            std::vector<uint16_t> fbuf((size_t)c->M_pad[l] * c->K_pad[l], 0);
            const uint16_t *src = (const uint16_t *)pol->weight[l];
            for (int m = 0; m < M; ++m)
                for (int k = 0; k < K; ++k) fbuf[im::frag_index(m, k, nks)] = src[(size_t)m * K + k];
            uint16_t *dwf = nullptr;
            IM_TRY_ALLOC(dwf, fbuf.size() * 2);
            c->d_wf.push_back(dwf);
            IM_TRY_HIP(hipMemcpy(dwf, fbuf.data(), fbuf.size() * 2, hipMemcpyHostToDevice),
                       "upload weights (fragment order)");
        }
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
        // large bf16 batches of the per-layer kernels stage the observation as
        // bf16 rows for the first layer (the one-launch kernel stages it in LDS)
        if (pol->dtype == IM_DTYPE_BF16 && max_envs > SMALL_BATCH && c->d_wf.empty())
            IM_TRY_ALLOC(c->d_obs16, (size_t)max_envs * (size_t)c->K_pad[0] * 2);
    }
    {
        // set-up of im_gae_noalloc's scratch on this device (its address is
        // looked up once per device, with the device current)
        double *scratch = nullptr;
        IM_TRY_HIP(im::gae_scratch_address(c->device, &scratch), "scratch address (hipGetSymbolAddress)");
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
    EnvArgs a = env_args(c, b);
    // threads per env: the configured split, or by batch size (path walks for
    // small batches, two halves up to SPLIT_ENV_MAX where a skeleton has no
    // path split, then one thread)
    int split = c->cfg.env_split;
    if (split == IM_SPLIT_AUTO)
        split = (a.n <= PATH_ENV_MAX && c->n_paths >= 2) ? IM_SPLIT_PATHS
                : (a.n <= SPLIT_ENV_MAX ? IM_SPLIT_HALVES : IM_SPLIT_ONE);
    int walk_slots = 0;
    a.n_parts = 1;
    if (split == IM_SPLIT_HALVES) {
        a.walks = c->d_skel->half;
        a.n_parts = 2;
        walk_slots = c->half_slots;
    } else if (split == IM_SPLIT_PATHS) {
        a.walks = c->d_skel->path;
        a.n_parts = c->n_paths;
        walk_slots = c->path_slots;
    }
    hipError_t e = launch_env_step(c->n_slots, walk_slots, a, (hipStream_t)stream);
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

}  // extern "C"

namespace {

// Checks of im_policy_act's arguments (context not null).
im_status check_act_args(const im_ctx *c, const float *obs, int64_t ld_obs, const uint32_t *env_n,
                         int64_t n_envs, const float *mean, const float *action)
{
    if (!obs || !env_n || !mean || !action) return fail(IM_ERR_INVALID_ARG, "NULL buffer");
    if (n_envs < 0 || n_envs > c->max_envs) return fail(IM_ERR_INVALID_ARG, "n_envs must be in [0, max_envs]");
    if (ld_obs < n_envs || ld_obs < 1) return fail(IM_ERR_INVALID_ARG, "ld_obs must be >= n_envs");
    return IM_OK;
}

// Extents of the policy's layer inputs: buffer loads address with 32-bit byte offsets.
im_status check_act_sizes(const im_ctx *c, int64_t ld_obs, int64_t n_envs)
{
    const bool bf16 = c->dtype == IM_DTYPE_BF16;
    const uint64_t esz = bf16 ? 2 : 4;
    for (int l = 0; l < c->L; ++l) {
        const uint64_t xb = l == 0 ? (uint64_t)c->D * (uint64_t)ld_obs * 4
                                   : (uint64_t)n_envs * (uint64_t)c->M_pad[l - 1] * esz;
        if (xb > 0xFFFFFFF0ull)
            return fail(IM_ERR_UNSUPPORTED, "policy input of layer " + std::to_string(l) +
                                                " exceeds 4 GiB");
    }
    if (c->d_obs16 && (uint64_t)n_envs * (uint64_t)c->K_pad[0] * 2 > 0xFFFFFFF0ull)
        return fail(IM_ERR_UNSUPPORTED, "staged policy input exceeds 4 GiB");
    return IM_OK;
}

// The policy's layers; *staged: the first layer read the observation through
// the bf16 staging buffer (which then holds it).
im_status policy_layers(im_ctx *c, const float *obs, int64_t ld_obs, const uint32_t *env_n,
                        int64_t n_envs, float *mean, float *action, float *logp,
                        hipStream_t stream, bool *staged)
{
    const bool bf16 = c->dtype == IM_DTYPE_BF16;
    const uint64_t esz = bf16 ? 2 : 4;
    if (bf16 && !c->d_wf.empty()) {
        FusedMlpArgs f{};
        f.obs = obs;
        f.ld_obs = ld_obs;
        f.obs_bytes = (uint32_t)((uint64_t)c->D * (uint64_t)ld_obs * 4);
        f.D = c->D;
        f.L = c->L;
        for (int l = 0; l < c->L; ++l) {
            f.w[l] = c->d_wf[l];
            f.bias[l] = c->d_b[l];
            f.w_bytes[l] = (uint32_t)((uint64_t)c->M_pad[l] * (uint64_t)c->K_pad[l] * 2);
            f.M_pad[l] = c->M_pad[l];
            f.K_pad[l] = c->K_pad[l];
        }
        GemmArgs &g = f.out;
        g.N = n_envs;
        g.bias = c->d_b[c->L - 1];
        g.mean = mean;
        g.action = action;
        g.logp = logp;
        g.env_n = env_n;
        g.log_std = c->d_log_std;
        g.A = c->A;
        g.seed = c->cfg.seed;
        hipError_t e = launch_policy_fused(f, stream);
        if (e != hipSuccess) return hip_fail(e, "fused policy launch");
        return IM_OK;
    }
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
        hipError_t e = launch_policy_layer(bf16, l == 0, last, g, c->M_pad[l], stream,
                                           l == 0 ? staged : nullptr);
        if (e != hipSuccess) return hip_fail(e, "policy layer launch");
    }
    return IM_OK;
}

}  // namespace

extern "C" {

im_status im_policy_act(im_ctx *c, const float *obs, int64_t ld_obs, const uint32_t *env_n,
                        int64_t n_envs, float *mean, float *action, float *logp, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    im_status s = check_act_args(c, obs, ld_obs, env_n, n_envs, mean, action);
    if (s != IM_OK) return s;
    if ((s = check_device(c)) != IM_OK) return s;
    if ((s = check_act_sizes(c, ld_obs, n_envs)) != IM_OK) return s;
    return policy_layers(c, obs, ld_obs, env_n, n_envs, mean, action, logp, (hipStream_t)stream,
                         nullptr);
}

}  // extern "C"

namespace {

// Hidden layers 0..n_hidden-1 of a packed MLP (bias, ReLU, the dtype's
// rounding) on the observation; the last activations end in d_ws[(n_hidden-1) & 1].
// staged: the bf16 staging buffer already holds this observation.
im_status mlp_hidden(im_ctx *c, int n_hidden, const std::vector<int> &M_pad,
                     const std::vector<int> &K_pad, const std::vector<void *> &d_w,
                     const std::vector<float *> &d_b, const float *obs, int64_t ld_obs,
                     int64_t n_envs, hipStream_t stream, bool staged)
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
        g.x16_staged = l == 0 && staged;
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
    // hidden layers of a bf16 critic that the one-launch kernel holds, again in
    // MFMA fragment order
    bool fits = bf16 && L >= 2 && L - 1 <= FUSED_MAX_LAYERS && cr.K_pad[0] <= FUSED_MAX_WIDTH;
    for (int l = 0; l < L - 1; ++l) fits = fits && cr.M_pad[l] <= FUSED_MAX_WIDTH;
    for (int l = 0; fits && l < L - 1; ++l) {
        const int M = cr.dims[l + 1], K = cr.dims[l], nks = cr.K_pad[l] / 64;
        std::vector<uint16_t> fbuf((size_t)cr.M_pad[l] * cr.K_pad[l], 0);
        const uint16_t *src = (const uint16_t *)k->weight[l];
        for (int m = 0; m < M; ++m)
            for (int i = 0; i < K; ++i) fbuf[im::frag_index(m, i, nks)] = src[(size_t)m * K + i];
        uint16_t *dwf = nullptr;
        if (!alloc(&dwf, fbuf.size() * 2)) return oom("critic weights (fragment order)");
        cr.d_wf.push_back(dwf);
        if ((e = hipMemcpy(dwf, fbuf.data(), fbuf.size() * 2, hipMemcpyHostToDevice)) != hipSuccess)
            return upload_fail(e, "upload critic weights (fragment order)");
    }
    // last layer as an fp32 vector (bf16 weights convert exactly)
    cr.K_head = L == 1 ? c->D : cr.M_pad[L - 2];
    std::vector<float> head(cr.K_head + 1, 0.0f);
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
    head[cr.K_head] = k->bias[L - 1][0];
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
        if (bf16 && c->max_envs > SMALL_BATCH && !c->d_obs16 && cr.d_wf.empty() &&
            dev_alloc(c, &c->d_obs16, (size_t)c->max_envs * (size_t)round_up(c->D, 64) * 2) !=
                hipSuccess)
            return oom("observation staging");
    }
    cr.L = L;
    return IM_OK;
}

}  // extern "C"

namespace {

// Checks of im_value's arguments (context not null).
im_status check_value_args(const im_ctx *c, const float *obs, int64_t ld_obs, int64_t n_envs,
                           const float *value)
{
    if (c->critic.L == 0) return fail(IM_ERR_INVALID_ARG, "no critic (im_set_critic)");
    if (!obs || !value) return fail(IM_ERR_INVALID_ARG, "NULL buffer");
    if (n_envs < 0 || n_envs > c->max_envs) return fail(IM_ERR_INVALID_ARG, "n_envs must be in [0, max_envs]");
    if (ld_obs < n_envs || ld_obs < 1) return fail(IM_ERR_INVALID_ARG, "ld_obs must be >= n_envs");
    return IM_OK;
}

im_status check_value_sizes(const im_ctx *c, int64_t ld_obs, int64_t n_envs)
{
    const auto &cr = c->critic;
    const uint64_t esz = c->dtype == IM_DTYPE_BF16 ? 2 : 4;
    if ((uint64_t)c->D * (uint64_t)ld_obs * 4 > 0xFFFFFFF0ull)
        return fail(IM_ERR_UNSUPPORTED, "critic input exceeds 4 GiB");
    for (int l = 1; l < cr.L - 1; ++l)
        if ((uint64_t)n_envs * (uint64_t)cr.M_pad[l - 1] * esz > 0xFFFFFFF0ull)
            return fail(IM_ERR_UNSUPPORTED, "critic layer input exceeds 4 GiB");
    if (c->d_obs16 && (uint64_t)n_envs * (uint64_t)round_up(c->D, 64) * 2 > 0xFFFFFFF0ull)
        return fail(IM_ERR_UNSUPPORTED, "staged critic input exceeds 4 GiB");
    return IM_OK;
}

// The critic's layers; staged: the bf16 staging buffer already holds obs.
im_status value_layers(im_ctx *c, const float *obs, int64_t ld_obs, int64_t n_envs, float *value,
                       hipStream_t st, bool staged)
{
    const auto &cr = c->critic;
    const bool bf16 = c->dtype == IM_DTYPE_BF16;
    hipError_t e;
    if (!cr.d_wf.empty()) {
        FusedMlpArgs f{};
        f.obs = obs;
        f.ld_obs = ld_obs;
        f.obs_bytes = (uint32_t)((uint64_t)c->D * (uint64_t)ld_obs * 4);
        f.D = c->D;
        f.L = cr.L - 1;
        for (int l = 0; l < f.L; ++l) {
            f.w[l] = cr.d_wf[l];
            f.bias[l] = cr.d_b[l];
            f.w_bytes[l] = (uint32_t)((uint64_t)cr.M_pad[l] * (uint64_t)cr.K_pad[l] * 2);
            f.M_pad[l] = cr.M_pad[l];
            f.K_pad[l] = cr.K_pad[l];
        }
        f.out.N = n_envs;
        f.head = cr.d_head;
        f.value = value;
        e = launch_value_fused(f, st);
        return e == hipSuccess ? IM_OK : hip_fail(e, "fused value launch");
    }
    if (cr.L == 1) {
        e = launch_value_head_obs(obs, ld_obs, c->D, cr.d_head, cr.d_head + cr.K_head, bf16, n_envs,
                                  value, st);
    } else {
        im_status s = mlp_hidden(c, cr.L - 1, cr.M_pad, cr.K_pad, cr.d_w, cr.d_b, obs, ld_obs,
                                 n_envs, st, staged);
        if (s != IM_OK) return s;
        e = launch_value_head_rows(bf16, c->d_ws[(cr.L - 2) & 1], cr.K_head, cr.K_head, cr.d_head,
                                   cr.d_head + cr.K_head, n_envs, value, st);
    }
    return e == hipSuccess ? IM_OK : hip_fail(e, "value head launch");
}

}  // namespace

extern "C" {

im_status im_value(im_ctx *c, const float *obs, int64_t ld_obs, int64_t n_envs, float *value,
                   void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    im_status s = check_value_args(c, obs, ld_obs, n_envs, value);
    if (s != IM_OK) return s;
    if ((s = check_device(c)) != IM_OK) return s;
    if ((s = check_value_sizes(c, ld_obs, n_envs)) != IM_OK) return s;
    return value_layers(c, obs, ld_obs, n_envs, value, (hipStream_t)stream, false);
}

im_status im_policy_act_value(im_ctx *c, const float *obs, int64_t ld_obs, const uint32_t *env_n,
                              int64_t n_envs, float *mean, float *action, float *logp,
                              float *value, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    im_status s = check_act_args(c, obs, ld_obs, env_n, n_envs, mean, action);
    if (s != IM_OK) return s;
    if ((s = check_value_args(c, obs, ld_obs, n_envs, value)) != IM_OK) return s;
    if ((s = check_device(c)) != IM_OK) return s;
    if ((s = check_act_sizes(c, ld_obs, n_envs)) != IM_OK) return s;
    if ((s = check_value_sizes(c, ld_obs, n_envs)) != IM_OK) return s;
    const hipStream_t st = (hipStream_t)stream;
    bool staged = false;
    if ((s = policy_layers(c, obs, ld_obs, env_n, n_envs, mean, action, logp, st, &staged)) != IM_OK)
        return s;
    return value_layers(c, obs, ld_obs, n_envs, value, st, staged);
}

}  // extern "C"

namespace {

// validation shared by im_gae and im_gae_noalloc; max_envs bounds n_envs
im_status check_rollout(const im_rollout *r, int64_t max_envs, im_status too_many, const char *limit)
{
    if (!r) return fail(IM_ERR_INVALID_ARG, "NULL rollout");
    if (r->T < 1) return fail(IM_ERR_INVALID_ARG, "T must be >= 1");
    if (r->n_envs < 0) return fail(IM_ERR_INVALID_ARG, "n_envs must be >= 0");
    if (r->n_envs > max_envs) return fail(too_many, std::string("n_envs above ") + limit);
    if (r->ld < r->n_envs || r->ld < 1) return fail(IM_ERR_INVALID_ARG, "ld must be >= n_envs and >= 1");
    if (!r->reward || !r->terminated || !r->truncated || !r->value || !r->advantage || !r->ret)
        return fail(IM_ERR_INVALID_ARG, "NULL rollout buffer");
    if (r->summary && (!r->ep_return || !r->ep_length))
        return fail(IM_ERR_INVALID_ARG, "summaries need ep_return and ep_length");
    if (!(r->gamma >= 0.0f && r->gamma <= 1.0f) || !(r->lambda >= 0.0f && r->lambda <= 1.0f))
        return fail(IM_ERR_INVALID_ARG, "gamma and lambda must be in [0, 1]");
    return IM_OK;
}

GaeArgs gae_args(const im_rollout *r, double *partial)
{
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
    g.partial = partial;
    return g;
}

}  // namespace

extern "C" {

im_status im_gae(im_ctx *c, const im_rollout *r, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    im_status s = check_rollout(r, c->max_envs, IM_ERR_INVALID_ARG, "max_envs");
    if (s != IM_OK) return s;
    s = check_device(c);
    if (s != IM_OK) return s;
    hipError_t e = launch_gae(gae_args(r, c->d_partial), (hipStream_t)stream);
    return e == hipSuccess ? IM_OK : hip_fail(e, "gae launch");
}

im_status im_gae_noalloc(const im_rollout *r, void *stream)
{
    im_status s = check_rollout(r, IM_GAE_NOALLOC_MAX_ENVS, IM_ERR_UNSUPPORTED,
                                "IM_GAE_NOALLOC_MAX_ENVS (the size of the call's scratch)");
    if (s != IM_OK) return s;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    double *scratch = nullptr;
    e = im::gae_scratch_address(dev, &scratch);
    if (e != hipSuccess) return hip_fail(e, "scratch address (hipGetSymbolAddress)");
    e = launch_gae(gae_args(r, scratch), (hipStream_t)stream);
    return e == hipSuccess ? IM_OK : hip_fail(e, "gae launch");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// PPO update: training state and entry points.
// ---------------------------------------------------------------------------
namespace im {

struct TrainLayer {
    int out = 0, in = 0, Mp = 0, Kp = 0;   // Mp, Kp: multiples of the 128 GEMM tile
    int64_t w_off = 0, b_off = 0;          // in the parameter vector
    uint16_t *wt = nullptr;                // [Mp][Kp] bf16
    uint16_t *wtt = nullptr;               // [Kp][Mp] bf16
    float *bias = nullptr;                 // [Mp]
    uint16_t *act = nullptr;               // hidden output [Mp][Mb] bf16 (null: output layer)
    uint4 *mbits = nullptr;                // its ReLU mask as bits, tile-major (Mp % 256 == 0)
    void *roll = nullptr;                  // the rollout's packed copy [.][roll_K]
    int roll_K = 0;
    uint16_t *rollf = nullptr;             // the rollout's fragment-order copy, or null
    float *roll_bias = nullptr;
};

struct TrainState {
    int64_t Mb_max = 0;                    // samples per minibatch, padded to 256
    int64_t P = 0;                         // parameters
    float *x = nullptr, *m = nullptr, *v = nullptr, *grad = nullptr;
    int *step = nullptr;
    OptScalars *opt = nullptr;
    std::vector<TrainLayer> actor, critic;  // critic: its hidden layers
    int64_t log_std_off = 0, head_w_off = 0, head_b_off = 0;
    int head_K = 0;                        // input width of the critic's output layer
    int Kp0 = 0;
    uint16_t *x0 = nullptr;                // [Kp0][Mb] gathered observation (bf16)
    float *act = nullptr, *mean_old = nullptr;   // [A][Mb]
    float *logp_old = nullptr, *adv = nullptr, *ret = nullptr, *vold = nullptr;
    float *mean_new = nullptr, *value_new = nullptr, *dv = nullptr;
    uint16_t *dmu = nullptr;               // [Mp of the actor's output layer][Mb], rows >= A zero
    uint16_t *dz[2] = {nullptr, nullptr};  // [max width][Mb]
    float *splitk = nullptr;
    size_t splitk_floats = 0;
    double *loss_partial = nullptr, *mb_stats = nullptr, *norm_partial = nullptr;
    double *rowsum_part = nullptr;         // [rows][segments] of the bias-gradient sums
    double *rs_tile = nullptr;             // [rows][column tiles]: row sums of a masked
                                           // gradient, left by the kernel that wrote it
    double *head_part = nullptr;           // [head_K][blocks]: the critic head's weight gradient
    int norm_blocks = 0;
    float *log_std_old = nullptr;
    int64_t last_Mbp = 0;                  // padded samples of the last minibatch run
    std::vector<void *> allocs;
    int64_t bytes = 0;
};

void free_train(TrainState *t)
{
    if (!t) return;
    for (void *p : t->allocs) hipFree(p);
    delete t;
}

}  // namespace im

namespace {

using im::TrainLayer;
using im::TrainState;

// split-K for a weight gradient of tiles x (K = Mb): about 1024 blocks, at
// least 4 K steps each
void splitk_plan(int tiles, int64_t Mb, int *splits, int *k_split)
{
    int64_t S = (1024 + tiles - 1) / tiles;
    const int64_t smax = Mb / 256 > 0 ? Mb / 256 : 1;
    if (S > smax) S = smax;
    if (S < 1) S = 1;
    int64_t ks = round_up((Mb + S - 1) / S, 64);
    *k_split = (int)ks;
    *splits = (int)((Mb + ks - 1) / ks);
}

im_status tg(bool bt, int epi, const im::TGemm &g, int splits, hipStream_t st)
{
    hipError_t e = im::launch_tgemm(bt, epi, g, splits, st);
    return e == hipSuccess ? IM_OK : hip_fail(e, "training GEMM launch");
}

#define IM_CHK(call)                                          \
    do {                                                      \
        hipError_t e_ = (call);                               \
        if (e_ != hipSuccess) return hip_fail(e_, #call);     \
    } while (0)
#define IM_CHS(call)                   \
    do {                               \
        im_status s_ = (call);         \
        if (s_ != IM_OK) return s_;    \
    } while (0)

// Whether a hidden layer's forward writes (and the next layer's input gradient
// reads) its ReLU mask as bits: 256x256 tiles only.
bool mbits_ok(const TrainLayer &L, int64_t Mb)
{
    return L.mbits && L.Mp % 256 == 0 && Mb % 256 == 0;
}

// forward of one network's GEMM layers; returns the output of the last one
im_status net_forward(const std::vector<TrainLayer> &net, const uint16_t *x0, int Kp0, int64_t Mb,
                      bool linear_last, float *out_last, int M_valid, hipStream_t st)
{
    const uint16_t *x = x0;
    int Kx = Kp0;
    for (size_t l = 0; l < net.size(); ++l) {
        const TrainLayer &L = net[l];
        const bool last = linear_last && l + 1 == net.size();
        im::TGemm g{};
        g.A = L.wt;
        g.lda = L.Kp;
        g.a_bytes = (uint32_t)((uint64_t)L.Mp * L.Kp * 2);
        g.B = x;
        g.ldb = Mb;
        g.b_bytes = (uint32_t)((uint64_t)Kx * Mb * 2);
        g.M = L.Mp;
        g.N = (int)Mb;
        g.K = L.Kp;
        g.k_split = L.Kp;
        g.bias = L.bias;
        g.ldc = Mb;
        if (last) {
            g.C = out_last;
            g.M_valid = M_valid;
            IM_CHS(tg(true, im::T_LINEAR, g, 1, st));
        } else {
            g.C = L.act;
            g.mbits = mbits_ok(L, Mb) ? L.mbits : nullptr;
            IM_CHS(tg(true, im::T_HIDDEN, g, 1, st));
        }
        x = L.act;
        Kx = L.Mp;
    }
    return IM_OK;
}

// Columns of a layer's weight-gradient GEMM: its input width padded to the
// 256-column tile.
int wgrad_cols(const TrainLayer &L) { return (int)round_up(L.Kp, 256); }

// backward of one network's GEMM layers from dz (gradient of the last GEMM
// layer's pre-activation, [Mp][Mb] bf16): weight and bias gradients into
// t->grad; dz buffers alternate in t->dz starting after `dz`
im_status net_backward(TrainState *t, const std::vector<TrainLayer> &net, const uint16_t *x0,
                       const uint16_t *dz, int64_t Mb, hipStream_t st, int top_parts = 0)
{
    int pp = dz == t->dz[0] ? 1 : 0;
    // dz came with its row sums in t->rs_tile, by `parts` column blocks: given
    // for the top layer (top_parts), then left by each masked-gradient GEMM
    bool dz_sums = top_parts > 0;
    int parts = top_parts;
    for (int l = (int)net.size() - 1; l >= 0; --l) {
        const TrainLayer &L = net[l];
        const uint16_t *X = l == 0 ? x0 : net[l - 1].act;
        // dW = dZ^T X over the minibatch (split over it), on whole 256-column tiles:
        // the columns past Kp read zero (outside the operand's buffer range)
        const int Nw = wgrad_cols(L);
        const int tiles = (L.Mp / 128) * (Nw / 128);
        int S, ks;
        splitk_plan(tiles, Mb, &S, &ks);
        im::TGemm g{};
        g.A = dz;
        g.lda = Mb;
        g.a_bytes = (uint32_t)((uint64_t)L.Mp * Mb * 2);
        g.B = X;
        g.ldb = Mb;
        g.b_bytes = (uint32_t)((uint64_t)L.Kp * Mb * 2);
        g.M = L.Mp;
        g.N = Nw;
        g.K = (int)Mb;
        g.k_split = ks;
        g.C = t->splitk;
        g.ldc = Nw;
        IM_CHS(tg(false, im::T_PARTIAL, g, S, st));
        IM_CHK(im::launch_splitk_reduce(t->splitk, S, L.Mp, Nw, L.out, L.in, t->grad + L.w_off, st));
        if (dz_sums)
            IM_CHK(im::launch_rowsum_finish(t->rs_tile, L.out, parts, t->grad + L.b_off, st));
        else
            IM_CHK(im::launch_rowsum(true, dz, L.out, Mb, nullptr, t->rowsum_part, t->grad + L.b_off, st));
        if (l == 0) break;
        // dX^T = W^T dZ^T, masked where the layer input (a ReLU output) is 0
        im::TGemm h{};
        h.A = L.wtt;
        h.lda = L.Mp;
        h.a_bytes = (uint32_t)((uint64_t)L.Kp * L.Mp * 2);
        h.B = dz;
        h.ldb = Mb;
        h.b_bytes = (uint32_t)((uint64_t)L.Mp * Mb * 2);
        h.M = L.Kp;
        h.N = (int)Mb;
        h.K = L.Mp;
        h.k_split = L.Mp;
        h.C = t->dz[pp];
        h.ldc = Mb;
        h.mask = X;
        h.ldm = Mb;
        // the mask bits the forward of layer l - 1 wrote on the same tiles
        if (mbits_ok(net[l - 1], Mb) && net[l - 1].Mp == L.Kp) h.mbits = net[l - 1].mbits;
        h.rs_part = t->rs_tile;     // the bias gradient of layer l - 1, by column tile
        IM_CHS(tg(true, im::T_MASK, h, 1, st));
        dz_sums = true;
        parts = (int)(Mb / im::tgemm_bn(Mb));
        dz = t->dz[pp];
        pp ^= 1;
    }
    return IM_OK;
}

// minibatch chunk range of (epoch, mb): numpy array_split of the epoch's chunks
void mb_range(int64_t n_chunks, int mbs, int mb, int64_t *first, int64_t *count)
{
    const int64_t q = n_chunks / mbs, r = n_chunks % mbs;
    *first = mb * q + (mb < r ? mb : r);
    *count = q + (mb < r ? 1 : 0);
}

// forward, loss and backward of one minibatch: t->grad and t->mb_stats
im_status run_minibatch(im_ctx *c, const im_ppo_batch *b, const im_ppo_params *p, int epoch, int mb,
                        hipStream_t st)
{
    TrainState *t = c->train;
    const int64_t n_chunks = (int64_t)b->T * (b->n_envs / 64);
    int64_t first, count;
    mb_range(n_chunks, p->minibatches, mb, &first, &count);
    const int64_t Mb = count * 64;
    const int64_t Mbp = round_up(Mb, 256);
    t->last_Mbp = Mbp;
    im::GatherArgs ga{};
    ga.obs = b->obs;
    ga.action = b->action;
    ga.mean = b->mean;
    ga.logp = b->logp;
    ga.adv_src = b->advantage;
    ga.ret_src = b->ret;
    ga.value = b->value;
    ga.perm = b->perm + (int64_t)epoch * n_chunks + first;
    ga.chunks = (int)count;
    ga.chunks_pad = (int)(Mbp / 64);
    ga.n_chunks = (int)n_chunks;
    ga.cpt = b->n_envs / 64;
    ga.N = b->n_envs;
    ga.ld = b->ld;
    ga.Mb_pad = Mbp;
    ga.D = c->D;
    ga.K0 = t->Kp0;
    ga.A = c->A;
    ga.x0 = t->x0;
    ga.act = t->act;
    ga.mean_old = t->mean_old;
    ga.logp_old = t->logp_old;
    ga.adv = t->adv;
    ga.ret = t->ret;
    ga.vold = t->vold;
    IM_CHK(im::launch_gather(ga, st));
    // forward
    IM_CHS(net_forward(t->actor, t->x0, t->Kp0, Mbp, true, t->mean_new, c->A, st));
    IM_CHS(net_forward(t->critic, t->x0, t->Kp0, Mbp, false, nullptr, 0, st));
    const TrainLayer &hl = t->critic.back();
    const float *head = c->critic.d_head;
    IM_CHK(im::launch_head_forward(hl.act, t->head_K, Mbp, head, head + c->critic.K_head, t->value_new,
                                   st));
    // loss
    im::LossArgs la{};
    la.Mb = Mb;
    la.Mb_pad = Mbp;
    la.A = c->A;
    la.n_samples = (int64_t)b->T * b->n_envs;
    la.summary = b->summary;
    la.mean = t->mean_new;
    la.act = t->act;
    la.mean_old = t->mean_old;
    la.log_std = t->x + t->log_std_off;
    la.log_std_old = t->log_std_old;
    la.logp_old = t->logp_old;
    la.adv = t->adv;
    la.ret = t->ret;
    la.vold = t->vold;
    la.value = t->value_new;
    la.clip = p->clip;
    la.value_coef = p->value_coef;
    la.clipped_value_loss = p->clipped_value_loss;
    la.dmu = t->dmu;
    la.dv = t->dv;
    la.partial = t->loss_partial;
    IM_CHK(im::launch_loss(la, st));
    im::LossReduceArgs lr{};
    lr.partial = t->loss_partial;
    lr.blocks = (int)(Mbp / 256);
    lr.A = c->A;
    lr.Mb = Mb;
    lr.entropy_coef = p->entropy_coef;
    lr.grad_log_std = t->grad + t->log_std_off;
    lr.mb_stats = t->mb_stats;
    IM_CHK(im::launch_loss_reduce(lr, st));
    // backward: actor from the output-layer gradient, critic from dV
    IM_CHS(net_backward(t, t->actor, t->x0, t->dmu, Mbp, st));
    IM_CHK(im::launch_rowsum(false, t->dv, 1, Mbp, nullptr, t->rowsum_part, t->grad + t->head_b_off, st));
    // the head's weight gradient and the top hidden layer's bias-gradient sums
    // come out of the kernel that forms that layer's gradient
    const int hparts = (int)((Mbp / 8 + 255) / 256);
    IM_CHK(im::launch_head_backward(hl.act, t->head_K, hl.Mp, Mbp, head, t->dv, t->dz[0], t->head_part,
                                    t->rs_tile, st));
    IM_CHK(im::launch_rowsum_finish(t->head_part, t->head_K, hparts, t->grad + t->head_w_off, st));
    IM_CHS(net_backward(t, t->critic, t->x0, t->dz[0], Mbp, st, hparts));
    return IM_OK;
}

// training and rollout copies of every layer from the masters
im_status repack_all(im_ctx *c, hipStream_t st)
{
    TrainState *t = c->train;
    for (auto *net : {&t->actor, &t->critic})
        for (const TrainLayer &L : *net) {
            im::RepackArgs r{};
            r.W = t->x + L.w_off;
            r.b = t->x + L.b_off;
            r.out = L.out;
            r.in = L.in;
            r.wt = L.wt;
            r.wtt = L.wtt;
            r.Mp = L.Mp;
            r.Kp = L.Kp;
            r.roll = L.roll;
            r.roll_K = L.roll_K;
            r.rollf = L.rollf;
            r.roll_bf16 = 1;
            r.bias_train = L.bias;
            r.bias_roll = L.roll_bias;
            IM_CHK(im::launch_repack(r, st));
        }
    // the critic's output layer (bf16-rounded weights, as the forward uses them)
    im::RepackArgs h{};
    h.W = t->x + t->head_w_off;
    h.b = t->x + t->head_b_off;
    h.out = 1;
    h.in = t->head_K;
    h.roll = c->critic.d_head;
    h.roll_K = 0;
    h.roll_bf16 = 2;
    h.bias_roll = c->critic.d_head + c->critic.K_head;
    IM_CHK(im::launch_repack(h, st));
    IM_CHK(hipMemcpyAsync(c->d_log_std, t->x + t->log_std_off, sizeof(float) * c->A,
                          hipMemcpyDeviceToDevice, st));
    return IM_OK;
}

im_status check_ppo(const im_ctx *c, const im_ppo_batch *b, const im_ppo_params *p)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    if (!b || !p) return fail(IM_ERR_INVALID_ARG, "NULL argument");
    if (!c->train) return fail(IM_ERR_INVALID_ARG, "no training state (im_ppo_setup)");
    if (b->T < 1) return fail(IM_ERR_INVALID_ARG, "T must be >= 1");
    if (b->n_envs < 64 || b->n_envs % 64) return fail(IM_ERR_INVALID_ARG, "n_envs must be a positive multiple of 64");
    if (b->ld < b->n_envs) return fail(IM_ERR_INVALID_ARG, "ld must be >= n_envs");
    if (!b->obs || !b->action || !b->mean || !b->logp || !b->value || !b->advantage || !b->ret ||
        !b->summary || !b->perm || !b->lr)
        return fail(IM_ERR_INVALID_ARG, "NULL batch buffer");
    if (p->epochs < 1 || p->minibatches < 1) return fail(IM_ERR_INVALID_ARG, "epochs and minibatches must be >= 1");
    const int64_t n_chunks = (int64_t)b->T * (b->n_envs / 64);
    if (p->minibatches > n_chunks) return fail(IM_ERR_INVALID_ARG, "more minibatches than 64-env chunks");
    const int64_t largest = (n_chunks + p->minibatches - 1) / p->minibatches * 64;
    if (round_up(largest, 256) > c->train->Mb_max)
        return fail(IM_ERR_UNSUPPORTED, "minibatch of " + std::to_string(largest) +
                                            " samples exceeds the im_ppo_setup size");
    const float vals[] = {p->clip, p->value_coef, p->entropy_coef, p->max_grad_norm, p->beta1, p->beta2,
                          p->eps, p->desired_kl, p->lr_min, p->lr_max};
    for (float v : vals)
        if (!finite_f(v)) return fail(IM_ERR_INVALID_ARG, "PPO parameters must be finite");
    if (!(p->clip > 0.0f) || p->value_coef < 0.0f || p->entropy_coef < 0.0f)
        return fail(IM_ERR_INVALID_ARG, "clip must be > 0 and the coefficients >= 0");
    if (!(p->beta1 >= 0.0f && p->beta1 < 1.0f) || !(p->beta2 >= 0.0f && p->beta2 < 1.0f) || !(p->eps > 0.0f))
        return fail(IM_ERR_INVALID_ARG, "Adam betas must be in [0, 1) and eps > 0");
    if (!(p->lr_min > 0.0f) || p->lr_min > p->lr_max) return fail(IM_ERR_INVALID_ARG, "need 0 < lr_min <= lr_max");
    return check_device(c);
}

}  // namespace

extern "C" {

im_status im_ppo_setup(im_ctx *c, int64_t max_minibatch)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    if (c->dtype != IM_DTYPE_BF16) return fail(IM_ERR_UNSUPPORTED, "the PPO update needs a bf16 policy");
    if (c->critic.L < 2) return fail(IM_ERR_INVALID_ARG, "the PPO update needs a critic with a hidden layer");
    if (max_minibatch < 64 || max_minibatch > ((int64_t)1 << 24))
        return fail(IM_ERR_INVALID_ARG, "max_minibatch must be in [64, 2^24]");
    {
        // The training GEMMs address their bf16 [rows][minibatch] operands with
        // 32-bit byte extents and offsets: every such buffer (rows = a layer
        // width padded to 128) must stay below 4 GiB.
        int64_t rows = round_up(c->D, 128);
        for (int l = 1; l <= c->L; ++l) rows = std::max(rows, round_up(c->dims[l], 128));
        for (int l = 1; l <= c->critic.L; ++l) rows = std::max(rows, round_up(c->critic.dims[l], 128));
        if ((uint64_t)rows * (uint64_t)round_up(max_minibatch, 256) * 2 >= ((uint64_t)1 << 32))
            return fail(IM_ERR_UNSUPPORTED, "minibatch of " + std::to_string(max_minibatch) +
                                                " samples: a training operand would reach 4 GiB");
    }
    im_status s = check_device(c);
    if (s != IM_OK) return s;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "synchronise before the training setup");
    im::free_train(c->train);
    c->train = nullptr;
    auto *t = new TrainState();
    const int64_t Mb = round_up(max_minibatch, 256);
    t->Mb_max = Mb;
    auto alloc = [&](auto **p, size_t bytes) {
        void *q = nullptr;
        if (hipMalloc(&q, bytes) != hipSuccess) return false;
        t->allocs.push_back(q);
        t->bytes += (int64_t)bytes;
        *p = (std::remove_reference_t<decltype(*p)>)q;
        return hipMemset(q, 0, bytes) == hipSuccess;
    };
    auto oom = [&]() {
        im::free_train(t);
        return fail(IM_ERR_OOM, "device allocation failed (training state)");
    };
    // layer tables and parameter offsets
    int64_t off = 0;
    auto layer = [&](int out, int in) {
        TrainLayer L;
        L.out = out;
        L.in = in;
        L.Mp = (int)round_up(out, 128);
        L.Kp = (int)round_up(in, 128);
        L.w_off = off;
        off += (int64_t)out * in;
        L.b_off = off;
        off += out;
        return L;
    };
    for (int l = 0; l < c->L; ++l) t->actor.push_back(layer(c->dims[l + 1], c->dims[l]));
    t->log_std_off = off;
    off += c->A;
    const auto &cr = c->critic;
    for (int l = 0; l < cr.L - 1; ++l) t->critic.push_back(layer(cr.dims[l + 1], cr.dims[l]));
    t->head_K = cr.dims[cr.L - 1];
    t->head_w_off = off;
    off += t->head_K;
    t->head_b_off = off;
    off += 1;
    t->P = off;
    t->Kp0 = (int)round_up(c->D, 128);
    int maxw = 0;
    for (auto *net : {&t->actor, &t->critic})
        for (const TrainLayer &L : *net) maxw = std::max({maxw, L.Mp, L.Kp});
    // allocations
    const size_t P = (size_t)t->P;
    if (!alloc(&t->x, 4 * P) || !alloc(&t->m, 4 * P) || !alloc(&t->v, 4 * P) || !alloc(&t->grad, 4 * P) ||
        !alloc(&t->step, sizeof(int)) || !alloc(&t->opt, sizeof(im::OptScalars)))
        return oom();
    size_t sk = 0;
    for (auto *net : {&t->actor, &t->critic}) {
        for (size_t l = 0; l < net->size(); ++l) {
            TrainLayer &L = (*net)[l];
            const bool out_layer = net == &t->actor && l + 1 == net->size();
            if (!alloc(&L.wt, (size_t)L.Mp * L.Kp * 2) || !alloc(&L.wtt, (size_t)L.Kp * L.Mp * 2) ||
                !alloc(&L.bias, sizeof(float) * L.Mp))
                return oom();
            if (!out_layer && !alloc(&L.act, (size_t)L.Mp * Mb * 2)) return oom();
            if (!out_layer && L.Mp % 256 == 0 && !alloc(&L.mbits, (size_t)L.Mp * Mb / 8)) return oom();
            int S, ks;
            splitk_plan((L.Mp / 128) * (wgrad_cols(L) / 128), Mb, &S, &ks);
            sk = std::max(sk, (size_t)S * L.Mp * wgrad_cols(L));
        }
    }
    const int A = c->A;
    const TrainLayer &al = t->actor.back();
    if (!alloc(&t->x0, (size_t)t->Kp0 * Mb * 2) || !alloc(&t->act, 4 * (size_t)A * Mb) ||
        !alloc(&t->mean_old, 4 * (size_t)A * Mb) || !alloc(&t->logp_old, 4 * (size_t)Mb) ||
        !alloc(&t->adv, 4 * (size_t)Mb) || !alloc(&t->ret, 4 * (size_t)Mb) || !alloc(&t->vold, 4 * (size_t)Mb) ||
        !alloc(&t->mean_new, 4 * (size_t)A * Mb) || !alloc(&t->value_new, 4 * (size_t)Mb) ||
        !alloc(&t->dv, 4 * (size_t)Mb) || !alloc(&t->dmu, (size_t)al.Mp * Mb * 2) ||
        !alloc(&t->dz[0], (size_t)maxw * Mb * 2) || !alloc(&t->dz[1], (size_t)maxw * Mb * 2) ||
        !alloc(&t->splitk, 4 * sk) ||
        !alloc(&t->loss_partial, sizeof(double) * (size_t)(Mb / 256) * (A + im::LOSS_STATS)) ||
        !alloc(&t->mb_stats, sizeof(double) * im::LOSS_STATS) || !alloc(&t->log_std_old, 4 * (size_t)A))
        return oom();
    t->splitk_floats = sk;
    t->norm_blocks = (int)std::min<int64_t>(1024, (t->P + 255) / 256);
    if (!alloc(&t->norm_partial, sizeof(double) * t->norm_blocks)) return oom();
    // row sums: rows x segments <= 2048 + rows for any row count
    if (!alloc(&t->rowsum_part, sizeof(double) * (2048 + (size_t)maxw + 1))) return oom();
    if (!alloc(&t->rs_tile, sizeof(double) * (size_t)maxw * (size_t)(Mb / 128 + 1))) return oom();
    if (!alloc(&t->head_part, sizeof(double) * (size_t)maxw * (size_t)(Mb / 2048 + 1))) return oom();
    // the rollout copies the update refreshes
    for (size_t l = 0; l < t->actor.size(); ++l) {
        t->actor[l].roll = c->d_w[l];
        t->actor[l].roll_K = c->K_pad[l];
        t->actor[l].rollf = c->d_wf.empty() ? nullptr : c->d_wf[l];
        t->actor[l].roll_bias = c->d_b[l];
    }
    for (size_t l = 0; l < t->critic.size(); ++l) {
        t->critic[l].roll = cr.d_w[l];
        t->critic[l].roll_K = cr.K_pad[l];
        t->critic[l].rollf = cr.d_wf.empty() ? nullptr : cr.d_wf[l];
        t->critic[l].roll_bias = cr.d_b[l];
    }
    // float32 masters from the current weights (bf16 values convert exactly)
    std::vector<float> x(P, 0.0f);
    auto unpack = [&](const void *dw, int M_pad_unused, int K_pad, const float *db, const TrainLayer &L) {
        (void)M_pad_unused;
        std::vector<uint16_t> w((size_t)L.out * K_pad);
        std::vector<float> bb(L.out);
        if (hipMemcpy(w.data(), dw, w.size() * 2, hipMemcpyDeviceToHost) != hipSuccess ||
            hipMemcpy(bb.data(), db, 4 * bb.size(), hipMemcpyDeviceToHost) != hipSuccess)
            return false;
        for (int o = 0; o < L.out; ++o)
            for (int i = 0; i < L.in; ++i) {
                const uint32_t u = (uint32_t)w[(size_t)o * K_pad + i] << 16;
                std::memcpy(&x[L.w_off + (int64_t)o * L.in + i], &u, 4);
            }
        std::memcpy(&x[L.b_off], bb.data(), 4 * bb.size());
        return true;
    };
    bool ok = true;
    for (size_t l = 0; l < t->actor.size() && ok; ++l)
        ok = unpack(c->d_w[l], c->M_pad[l], c->K_pad[l], c->d_b[l], t->actor[l]);
    for (size_t l = 0; l < t->critic.size() && ok; ++l)
        ok = unpack(cr.d_w[l], cr.M_pad[l], cr.K_pad[l], cr.d_b[l], t->critic[l]);
    ok = ok && hipMemcpy(&x[t->log_std_off], c->d_log_std, 4 * (size_t)A, hipMemcpyDeviceToHost) == hipSuccess;
    ok = ok && hipMemcpy(&x[t->head_w_off], cr.d_head, 4 * (size_t)t->head_K, hipMemcpyDeviceToHost) == hipSuccess;
    ok = ok && hipMemcpy(&x[t->head_b_off], cr.d_head + cr.K_head, 4, hipMemcpyDeviceToHost) == hipSuccess;
    ok = ok && hipMemcpy(t->x, x.data(), 4 * P, hipMemcpyHostToDevice) == hipSuccess;
    if (!ok) {
        im::free_train(t);
        return fail(IM_ERR_HIP, "initialise the master weights");
    }
    c->train = t;
    s = repack_all(c, nullptr);
    if (s == IM_OK && (e = hipDeviceSynchronize()) != hipSuccess) s = hip_fail(e, "training setup");
    if (s != IM_OK) {
        im::free_train(c->train);
        c->train = nullptr;
    }
    return s;
}

im_status im_ppo_update(im_ctx *c, const im_ppo_batch *b, const im_ppo_params *p, void *stream)
{
    im_status s = check_ppo(c, b, p);
    if (s != IM_OK) return s;
    TrainState *t = c->train;
    const hipStream_t st = (hipStream_t)stream;
    IM_CHK(hipMemcpyAsync(t->log_std_old, t->x + t->log_std_off, 4 * (size_t)c->A,
                          hipMemcpyDeviceToDevice, st));
    im::FinalizeArgs f{};
    f.norm_partial = t->norm_partial;
    f.norm_blocks = t->norm_blocks;
    f.mb_stats = t->mb_stats;
    f.max_grad_norm = p->max_grad_norm;
    f.desired_kl = p->desired_kl;
    f.lr_min = p->lr_min;
    f.lr_max = p->lr_max;
    f.beta1 = p->beta1;
    f.beta2 = p->beta2;
    f.eps = p->eps;
    f.lr = b->lr;
    f.step = t->step;
    f.opt = t->opt;
    f.stats = b->stats;
    for (int ep = 0; ep < p->epochs; ++ep)
        for (int mb = 0; mb < p->minibatches; ++mb) {
            IM_CHS(run_minibatch(c, b, p, ep, mb, st));
            IM_CHK(im::launch_optimizer(t->grad, t->P, t->norm_partial, t->norm_blocks, f, t->x, t->m, t->v, st));
            IM_CHS(repack_all(c, st));
        }
    return IM_OK;
}

im_status im_ppo_grad(im_ctx *c, const im_ppo_batch *b, const im_ppo_params *p, int32_t epoch,
                      int32_t minibatch, float *grad, double *stats, void *stream)
{
    im_status s = check_ppo(c, b, p);
    if (s != IM_OK) return s;
    if (!grad) return fail(IM_ERR_INVALID_ARG, "NULL gradient buffer");
    if (epoch < 0 || epoch >= p->epochs || minibatch < 0 || minibatch >= p->minibatches)
        return fail(IM_ERR_INVALID_ARG, "epoch or minibatch out of range");
    TrainState *t = c->train;
    const hipStream_t st = (hipStream_t)stream;
    IM_CHK(hipMemcpyAsync(t->log_std_old, t->x + t->log_std_off, 4 * (size_t)c->A,
                          hipMemcpyDeviceToDevice, st));
    IM_CHS(run_minibatch(c, b, p, epoch, minibatch, st));
    IM_CHK(hipMemcpyAsync(grad, t->grad, 4 * (size_t)t->P, hipMemcpyDeviceToDevice, st));
    if (stats)
        IM_CHK(hipMemcpyAsync(stats, t->mb_stats, sizeof(double) * im::LOSS_STATS,
                              hipMemcpyDeviceToDevice, st));
    return IM_OK;
}

im_status im_ppo_read(im_ctx *c, int32_t buffer, int32_t layer, void *dst, int64_t *rows,
                      int64_t *cols, int64_t *elem_bytes, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    const TrainState *t = c->train;
    if (!t) return fail(IM_ERR_INVALID_ARG, "no training state (im_ppo_setup)");
    if (t->last_Mbp <= 0) return fail(IM_ERR_INVALID_ARG, "no minibatch has run yet");
    if (buffer < 0 || buffer >= IM_PPO_BUFFERS) return fail(IM_ERR_INVALID_ARG, "unknown buffer");
    const bool hidden = buffer == IM_PPO_BUF_ACTOR_HIDDEN || buffer == IM_PPO_BUF_CRITIC_HIDDEN;
    if (!hidden && layer != 0) return fail(IM_ERR_INVALID_ARG, "layer must be 0 for this buffer");
    const void *src = nullptr;
    int64_t r = 0, eb = 2;
    switch (buffer) {
        case IM_PPO_BUF_INPUT: src = t->x0; r = t->Kp0; break;
        case IM_PPO_BUF_ACTOR_HIDDEN:
        case IM_PPO_BUF_CRITIC_HIDDEN: {
            const auto &net = buffer == IM_PPO_BUF_ACTOR_HIDDEN ? t->actor : t->critic;
            // the actor's last layer is its output, not a hidden layer
            const int n_hidden = (int)net.size() - (buffer == IM_PPO_BUF_ACTOR_HIDDEN ? 1 : 0);
            if (layer < 0 || layer >= n_hidden) return fail(IM_ERR_INVALID_ARG, "layer out of range");
            src = net[layer].act;
            r = net[layer].Mp;
            break;
        }
        case IM_PPO_BUF_MEAN: src = t->mean_new; r = c->A; eb = 4; break;
        case IM_PPO_BUF_VALUE: src = t->value_new; r = 1; eb = 4; break;
        case IM_PPO_BUF_DMEAN: src = t->dmu; r = t->actor.back().Mp; break;
        default: src = t->dv; r = 1; eb = 4; break;
    }
    if (rows) *rows = r;
    if (cols) *cols = t->last_Mbp;
    if (elem_bytes) *elem_bytes = eb;
    if (dst)
        IM_CHK(hipMemcpyAsync(dst, src, (size_t)(r * t->last_Mbp * eb), hipMemcpyDeviceToDevice,
                              (hipStream_t)stream));
    return IM_OK;
}

im_status im_ppo_params_get(im_ctx *c, float *params, int64_t *n, void *stream)
{
    if (!c) return fail(IM_ERR_INVALID_ARG, "NULL context");
    if (!c->train) return fail(IM_ERR_INVALID_ARG, "no training state (im_ppo_setup)");
    if (n) *n = c->train->P;
    if (params)
        IM_CHK(hipMemcpyAsync(params, c->train->x, 4 * (size_t)c->train->P, hipMemcpyDeviceToDevice,
                              (hipStream_t)stream));
    return IM_OK;
}

}  // extern "C"
#undef IM_CHK
#undef IM_CHS
