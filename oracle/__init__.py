"""ctypes front end of the CPU oracle (oracle/oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
CPU-baseline leg of the benchmark, never by the product package.  It shares
nothing with the HIP path; both consume the same seeded inputs.
"""
import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# IM_ORACLE_LIB selects another build of oracle.c (e.g. the sanitizer build of
# build.py --sanitize, run with the sanitizer runtime preloaded)
_LIB_PATH = os.environ.get("IM_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(np.uint32, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(np.uint8, flags="C_CONTIGUOUS")


def _opt(ptype):
    """Pointer argument that may be None."""
    class _Opt:
        @classmethod
        def from_param(cls, obj):
            if obj is None:
                return None
            return ptype.from_param(obj)
    return _Opt


_i64p_opt = _opt(np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS"))
_u8p_opt = _opt(_u8p)
_i32p_opt = _opt(_i32p)
_f32p_opt = _opt(_f32p)


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    L = C.CDLL(_LIB_PATH)
    L.or_philox.argtypes = [_u32p, _u32p, _u32p]
    L.or_normals.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint32, _f64p]
    for name in ("or_qmul",):
        getattr(L, name).argtypes = [_f64p, _f64p, _f64p]
    L.or_qrot.argtypes = [_f64p, _f64p, _f64p]
    L.or_rotvec.argtypes = [_f64p, _f64p]
    L.or_qexp.argtypes = [_f64p, _f64p]
    L.or_slerp.argtypes = [_f64p, _f64p, C.c_double, _f64p]
    L.or_round_bf16.argtypes = [C.c_double]
    L.or_round_bf16.restype = C.c_double
    L.or_world_create.argtypes = [
        C.c_int, _i32p, _i32p, _f32p, _f32p, _f32p, C.c_int, _i32p, _f32p, _f32p, _f32p, _f32p,
        C.c_double, C.c_float, C.c_float, C.c_int, _f32p, C.c_uint64]
    L.or_world_create.restype = C.c_void_p
    L.or_world_destroy.argtypes = [C.c_void_p]
    L.or_clip_dphi.argtypes = [C.c_void_p, C.c_int]
    L.or_clip_dphi.restype = C.c_float
    L.or_phase_index.argtypes = [C.c_int, C.c_float, C.POINTER(C.c_int), C.POINTER(C.c_float)]
    L.or_ref_state.argtypes = [C.c_void_p, C.c_int, C.c_float, _f64p, _f64p, _f64p, _f64p]
    L.or_fk.argtypes = [C.c_void_p, _f64p, _f64p, _f64p, _f64p, _f64p, _f64p, _f64p, _f64p, _f64p,
                        _f64p]
    L.or_reward.argtypes = [C.c_void_p, _f64p, _f64p, _f64p, _f64p, _f64p]
    L.or_terminated.argtypes = [C.c_void_p, C.c_int, C.c_float, C.c_float]
    L.or_terminated.restype = C.c_int
    L.or_obs.argtypes = [C.c_void_p, _f64p, _f64p, _f64p, _f64p, C.c_float, _f64p]
    L.or_reset_draw.argtypes = [C.c_void_p, C.c_uint32, C.c_uint32, C.c_uint32,
                                C.POINTER(C.c_int), C.POINTER(C.c_float)]
    L.or_env_step.argtypes = [
        C.c_void_p, C.c_int64, _i64p_opt, C.c_int64, _i32p, _f32p, _i32p, _u32p,
        _f32p, _f32p, _f32p, _f32p, C.c_int64, _f32p, _u8p, _u8p, _f32p, C.c_int64, _i32p_opt,
        _f32p_opt]
    L.or_world_set_training.argtypes = [C.c_void_p, C.c_int, _f32p, C.c_int, C.c_int, C.c_int]
    L.or_obs_dim.argtypes = [C.c_void_p]
    L.or_obs_dim.restype = C.c_int
    L.or_mreward.argtypes = [C.c_void_p, _f64p, _f64p, _f64p, C.c_int, C.c_float, _f64p]
    L.or_reset_envs.argtypes = [
        C.c_void_p, C.c_int64, _u8p_opt, _i32p, _f32p, _i32p, _u32p, _f32p, _f32p, _f32p, _f32p,
        C.c_int64, _f32p, C.c_int64]
    L.or_standin.argtypes = [
        C.c_void_p, C.c_int64, _i64p_opt, C.c_int64, _i32p, _f32p, _u32p, C.c_float, C.c_float,
        _f32p, _f32p, _f32p, _f32p, C.c_int64]
    L.or_policy.argtypes = [
        C.c_int, _i32p, C.c_int, _f32p, _f32p, _f32p, C.c_uint64, C.c_int64, _f32p, C.c_int64,
        _u32p, _i64p_opt, C.c_int64, _f32p, _f32p, _f32p_opt]
    L.or_num_threads.argtypes = []
    L.or_num_threads.restype = C.c_int
    _lib = L
    return L


def num_threads():
    return int(lib().or_num_threads())


# ---------------------------------------------------------------- primitives
def philox(ctr, key):
    out = np.zeros(4, np.uint32)
    lib().or_philox(np.asarray(ctr, np.uint32), np.asarray(key, np.uint32), out)
    return out


def normals(seed, e, n, block, tag):
    z = np.zeros(4, np.float64)
    lib().or_normals(seed, e, n, block, tag, z)
    return z


def qmul(a, b):
    out = np.zeros(4)
    lib().or_qmul(np.asarray(a, np.float64), np.asarray(b, np.float64), out)
    return out


def qrot(q, v):
    out = np.zeros(3)
    lib().or_qrot(np.asarray(q, np.float64), np.asarray(v, np.float64), out)
    return out


def rotvec(q):
    out = np.zeros(3)
    lib().or_rotvec(np.asarray(q, np.float64), out)
    return out


def qexp(r):
    out = np.zeros(4)
    lib().or_qexp(np.asarray(r, np.float64), out)
    return out


def slerp(a, b, t):
    out = np.zeros(4)
    lib().or_slerp(np.asarray(a, np.float64), np.asarray(b, np.float64), float(t), out)
    return out


def round_bf16(x):
    return lib().or_round_bf16(float(x))


def phase_index(F, phi):
    i0 = C.c_int()
    a = C.c_float()
    lib().or_phase_index(int(F), float(np.float32(phi)), C.byref(i0), C.byref(a))
    return i0.value, np.float32(a.value)


# ---------------------------------------------------------------- world
class World:
    """Oracle copy of a synthetic world (skeleton, clips, step configuration).

    `desc` is the dict made by paper_2609_09821_amd.synth.make_world.
    """

    def __init__(self, desc):
        sk = desc["skeleton"]
        clips = desc["clips"]
        cfg = desc["config"]
        self.B = int(sk["n_bodies"])
        self.n_clips = len(clips)
        self._keep = []

        def k(a, dt):
            a = np.ascontiguousarray(a, dtype=dt)
            self._keep.append(a)
            return a

        F = k([c["n_frames"] for c in clips], np.int32)
        fps = k([c["fps"] for c in clips], np.float32)
        rp = k(np.concatenate([c["root_pos"].reshape(-1) for c in clips]), np.float32)
        rq = k(np.concatenate([c["root_quat"].reshape(-1) for c in clips]), np.float32)
        lq = k(np.concatenate([c["local_quat"].reshape(-1) for c in clips]), np.float32)
        weights = k([cfg["c_pose"], cfg["w_pos"], cfg["w_ee"], cfg["c_vel"], cfg["w_vel"],
                     cfg["c_com"], cfg["w_com"]], np.float32)
        self.seed = int(cfg["seed"])
        self.ptr = lib().or_world_create(
            self.B, k(sk["parent"], np.int32), k(sk["jtype"], np.int32),
            k(sk["axis"], np.float32), k(sk["offset"], np.float32), k(sk["mass"], np.float32),
            self.n_clips, F, fps, rp, rq, lq, float(cfg["dt"]), float(cfg["h_term"]),
            float(cfg["r_min"]), int(cfg["grace"]), weights, self.seed)
        if not self.ptr:
            raise ValueError("oracle rejected the world description")
        self.A = int(desc["policy"]["dims"][-1])
        mw = k([cfg.get("m_jrot", 0.0), cfg.get("m_jvel", 0.0), cfg.get("m_com", 0.0),
                cfg.get("m_eepos", 0.0), cfg.get("m_eerot", 0.0)], np.float32)
        lib().or_world_set_training(self.ptr, int(cfg.get("reward_form", 0)), mw,
                                    int(cfg.get("obs_future", 0)),
                                    int(cfg.get("obs_prev_action", 0)), self.A)
        self.D = int(lib().or_obs_dim(self.ptr))

    def __del__(self):
        # at interpreter shutdown the module's globals may already be gone
        if getattr(self, "ptr", None) and lib is not None:
            lib().or_world_destroy(self.ptr)
            self.ptr = None

    # -- pins
    def dphi(self, k):
        return np.float32(lib().or_clip_dphi(self.ptr, int(k)))

    def ref_state(self, k, phi_ev):
        B = self.B
        P, Q, V, W = np.zeros(3 * B), np.zeros(4 * B), np.zeros(3 * B), np.zeros(3 * B)
        lib().or_ref_state(self.ptr, int(k), float(np.float32(phi_ev)), P, Q, V, W)
        return P.reshape(B, 3), Q.reshape(B, 4), V.reshape(B, 3), W.reshape(B, 3)

    def fk(self, root_p, root_q, root_v, root_w, q_local, w_local):
        B = self.B
        P, Q, V, W = np.zeros(3 * B), np.zeros(4 * B), np.zeros(3 * B), np.zeros(3 * B)
        f = lambda a: np.ascontiguousarray(a, np.float64).reshape(-1)
        lib().or_fk(self.ptr, f(root_p), f(root_q), f(root_v), f(root_w), f(q_local), f(w_local),
                    P, Q, V, W)
        return P.reshape(B, 3), Q.reshape(B, 4), V.reshape(B, 3), W.reshape(B, 3)

    def reward(self, P, V, Pr, Vr):
        out = np.zeros(5)
        f = lambda a: np.ascontiguousarray(a, np.float64).reshape(-1)
        lib().or_reward(self.ptr, f(P), f(V), f(Pr), f(Vr), out)
        return dict(e_pos=out[0], e_vel=out[1], e_ee=out[2], e_com=out[3], r=out[4])

    def mreward(self, P, Q, W, k, phi_ev):
        """Multiplicative reward terms of a sim state against clip k at phi_ev."""
        out = np.zeros(6)
        f = lambda a: np.ascontiguousarray(a, np.float64).reshape(-1)
        lib().or_mreward(self.ptr, f(P), f(Q), f(W), int(k), float(np.float32(phi_ev)), out)
        return dict(e_jrot=out[0], e_jvel=out[1], e_com=out[2], e_eepos=out[3], e_eerot=out[4],
                    r=out[5])

    def state(self, N):
        return State(self.B, N, self.D)

    def terminated(self, t_next, z_root, r_out):
        return bool(lib().or_terminated(self.ptr, int(t_next), float(np.float32(z_root)),
                                        float(np.float32(r_out))))

    def obs(self, P, Q, V, W, phase):
        out = np.zeros(15 * self.B + 1)
        f = lambda a: np.ascontiguousarray(a, np.float64).reshape(-1)
        lib().or_obs(self.ptr, f(P), f(Q), f(V), f(W), float(np.float32(phase)), out)
        return out

    def reset_draw(self, e, n, tag):
        kk = C.c_int()
        ph = C.c_float()
        lib().or_reset_draw(self.ptr, int(e), int(n), int(tag), C.byref(kk), C.byref(ph))
        return kk.value, np.float32(ph.value)

    # -- batch operations on State objects (numpy SoA buffers)
    def env_step(self, st, idx=None, prev_action=None):
        """prev_action: [N][A] float32, the actions applied in this step (needed when the
        observation holds the previous action)."""
        idx_a = None if idx is None else np.ascontiguousarray(idx, np.int64)
        pa = None if prev_action is None else np.ascontiguousarray(prev_action, np.float32)
        if pa is not None:
            assert pa.shape == (st.N, self.A)
        assert st.obs.shape[0] == self.D
        lib().or_env_step(self.ptr, st.N, idx_a, 0 if idx_a is None else len(idx_a),
                          st.clip, st.phase, st.t, st.n, st.pos, st.quat, st.linvel, st.angvel,
                          st.ld, st.reward, st.terminated, st.truncated, st.obs, st.ld,
                          st.ref_frame, pa)

    def reset_envs(self, st, mask=None):
        assert st.obs.shape[0] == self.D
        m = None if mask is None else np.ascontiguousarray(mask, np.uint8)
        lib().or_reset_envs(self.ptr, st.N, m, st.clip, st.phase, st.t, st.n, st.pos, st.quat,
                            st.linvel, st.angvel, st.ld, st.obs, st.ld)

    def standin(self, st, sigma_joint, sigma_vel, idx=None):
        idx_a = None if idx is None else np.ascontiguousarray(idx, np.int64)
        lib().or_standin(self.ptr, st.N, idx_a, 0 if idx_a is None else len(idx_a), st.clip,
                         st.phase, st.n, float(sigma_joint), float(sigma_vel), st.pos, st.quat,
                         st.linvel, st.angvel, st.ld)


class State:
    """Host SoA buffers in the library's layout (ld = N)."""

    def __init__(self, B, N, D=None):
        self.B, self.N, self.ld = B, N, N
        D = 15 * B + 1 if D is None else D
        self.clip = np.zeros(N, np.int32)
        self.phase = np.zeros(N, np.float32)
        self.t = np.zeros(N, np.int32)
        self.n = np.zeros(N, np.uint32)
        self.pos = np.zeros((B, 3, N), np.float32)
        self.quat = np.zeros((B, 4, N), np.float32)
        self.linvel = np.zeros((B, 3, N), np.float32)
        self.angvel = np.zeros((B, 3, N), np.float32)
        self.reward = np.zeros(N, np.float32)
        self.terminated = np.zeros(N, np.uint8)
        self.truncated = np.zeros(N, np.uint8)
        self.obs = np.zeros((D, N), np.float32)
        self.ref_frame = np.zeros(N, np.int32)

    def copy(self):
        s = State.__new__(State)
        for k, v in self.__dict__.items():
            s.__dict__[k] = v.copy() if isinstance(v, np.ndarray) else v
        return s


def policy(pol, seed, obs, env_n, idx=None):
    """Oracle policy forward + sampling.

    pol: dict from synth.make_policy (dims, bf16, W list, b list, log_std).
    obs: [D][N] float32; env_n: [N] uint32.  Returns mean, action [N][A], logp [N]
    (rows outside idx are left zero).
    """
    dims = np.asarray(pol["dims"], np.int32)
    L = len(dims) - 1
    Wall = np.ascontiguousarray(np.concatenate([w.reshape(-1) for w in pol["W"]]), np.float32)
    ball = np.ascontiguousarray(np.concatenate([b.reshape(-1) for b in pol["b"]]), np.float32)
    log_std = np.ascontiguousarray(pol["log_std"], np.float32)
    obs = np.ascontiguousarray(obs, np.float32)
    N = obs.shape[1]
    A = int(dims[-1])
    mean = np.zeros((N, A), np.float32)
    action = np.zeros((N, A), np.float32)
    logp = np.zeros(N, np.float32)
    idx_a = None if idx is None else np.ascontiguousarray(idx, np.int64)
    lib().or_policy(L, dims, int(bool(pol["bf16"])), Wall, ball, log_std, int(seed), N, obs, N,
                    np.ascontiguousarray(env_n, np.uint32), idx_a,
                    0 if idx_a is None else len(idx_a), mean, action, logp)
    return mean, action, logp


def value(critic, obs, idx=None):
    """Oracle value head: the critic MLP (same layer rules as the policy: ReLU
    hidden layers, bf16 rounding of the input and hidden activations for bf16
    critics, linear last layer of width 1) evaluated by the policy forward
    above with a zero log-std; the sampled part is discarded.

    critic: dict like synth.make_policy with dims[-1] == 1; obs: [D][N] float32.
    Returns value [N] float32 (entries outside idx are zero)."""
    assert critic["dims"][-1] == 1
    c = dict(critic)
    c["log_std"] = np.zeros(1, np.float32)
    N = np.asarray(obs).shape[1]
    mean, _, _ = policy(c, 0, obs, np.zeros(N, np.uint32), idx=idx)
    return mean[:, 0].copy()


from .rollout import gae, rollout_summary, SUMMARY_FIELDS  # noqa: E402
