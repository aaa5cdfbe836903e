"""ctypes binding of libinstantmimic.so (C ABI in include/instantmimic.h).

Argument marshalling only: every stage of the step runs in the HIP kernels of
the library.  PyTorch supplies device memory and the stream handle.  There is
no fallback: if the library is not built, loading raises.

Module-level functions carry the C names (im_create, im_env_step_fused,
im_policy_act, im_reset_envs, ...).  `Context` and `EnvBuffers` are small
conveniences over them for tensors.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libinstantmimic.so")

IM_OK, IM_ERR_INVALID_ARG, IM_ERR_UNSUPPORTED, IM_ERR_OOM, IM_ERR_HIP = range(5)
IM_DTYPE_F32, IM_DTYPE_BF16 = 0, 1
IM_GAE_NOALLOC_MAX_ENVS = 1 << 20   # im_gae_noalloc scratch limit
IM_JOINT_FREE, IM_JOINT_SPHERICAL, IM_JOINT_REVOLUTE, IM_JOINT_FIXED = range(4)
IM_SPLIT_AUTO, IM_SPLIT_ONE, IM_SPLIT_HALVES, IM_SPLIT_PATHS = range(4)


class ImConfig(C.Structure):
    _fields_ = [("dt", C.c_double), ("h_term", C.c_float), ("r_min", C.c_float),
                ("grace", C.c_int32), ("c_pose", C.c_float), ("w_pos", C.c_float),
                ("w_ee", C.c_float), ("c_vel", C.c_float), ("w_vel", C.c_float),
                ("c_com", C.c_float), ("w_com", C.c_float), ("seed", C.c_uint64),
                ("reward_form", C.c_int32), ("m_jrot", C.c_float), ("m_jvel", C.c_float),
                ("m_com", C.c_float), ("m_eepos", C.c_float), ("m_eerot", C.c_float),
                ("obs_future", C.c_int32), ("obs_prev_action", C.c_int32),
                ("env_split", C.c_int32)]


class ImSkeleton(C.Structure):
    _fields_ = [("n_bodies", C.c_int32), ("parent", C.POINTER(C.c_int32)),
                ("jtype", C.POINTER(C.c_int32)), ("axis", C.POINTER(C.c_float)),
                ("offset", C.POINTER(C.c_float)), ("mass", C.POINTER(C.c_float))]


class ImClip(C.Structure):
    _fields_ = [("n_frames", C.c_int32), ("fps", C.c_float), ("root_pos", C.POINTER(C.c_float)),
                ("root_quat", C.POINTER(C.c_float)), ("local_quat", C.POINTER(C.c_float))]


class ImPolicy(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("dims", C.POINTER(C.c_int32)), ("dtype", C.c_int32),
                ("weight", C.POINTER(C.c_void_p)), ("bias", C.POINTER(C.POINTER(C.c_float))),
                ("log_std", C.POINTER(C.c_float))]


class ImEnvBufs(C.Structure):
    _fields_ = [("body_pos", C.c_void_p), ("body_quat", C.c_void_p), ("body_linvel", C.c_void_p),
                ("body_angvel", C.c_void_p), ("env_clip", C.c_void_p), ("env_phase", C.c_void_p),
                ("env_t", C.c_void_p), ("env_n", C.c_void_p), ("reward", C.c_void_p),
                ("terminated", C.c_void_p), ("truncated", C.c_void_p), ("obs", C.c_void_p),
                ("ref_frame", C.c_void_p), ("n_envs", C.c_int64), ("ld", C.c_int64),
                ("prev_action", C.c_void_p)]


class ImRollout(C.Structure):
    _fields_ = [("T", C.c_int32), ("n_envs", C.c_int64), ("ld", C.c_int64), ("gamma", C.c_float),
                ("lam", C.c_float), ("reward", C.c_void_p), ("terminated", C.c_void_p),
                ("truncated", C.c_void_p), ("value", C.c_void_p), ("advantage", C.c_void_p),
                ("ret", C.c_void_p), ("ep_return", C.c_void_p), ("ep_length", C.c_void_p),
                ("summary", C.c_void_p)]


# fields of the rollout summary (IM_SUM_* order)
SUMMARY_FIELDS = ("reward_sum", "n_terminated", "n_truncated", "n_episodes",
                  "episode_return_sum", "episode_length_sum", "advantage_sum",
                  "advantage_sq_sum", "value_sum", "return_sum")


class ImPpoParams(C.Structure):
    _fields_ = [("clip", C.c_float), ("value_coef", C.c_float), ("entropy_coef", C.c_float),
                ("clipped_value_loss", C.c_int32), ("max_grad_norm", C.c_float),
                ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("desired_kl", C.c_float), ("lr_min", C.c_float), ("lr_max", C.c_float),
                ("epochs", C.c_int32), ("minibatches", C.c_int32)]


class ImPpoBatch(C.Structure):
    _fields_ = [("T", C.c_int32), ("n_envs", C.c_int64), ("ld", C.c_int64), ("obs", C.c_void_p),
                ("action", C.c_void_p), ("mean", C.c_void_p), ("logp", C.c_void_p),
                ("value", C.c_void_p), ("advantage", C.c_void_p), ("ret", C.c_void_p),
                ("summary", C.c_void_p), ("perm", C.c_void_p), ("lr", C.c_void_p),
                ("stats", C.c_void_p)]


# PPO update statistics (IM_PPO_* order)
PPO_STATS = ("loss_pi", "loss_v", "kl", "clip_frac", "grad_norm", "minibatches", "lr")
# im_ppo_read buffers (IM_PPO_BUF_*)
PPO_BUFFERS = ("input", "actor_hidden", "critic_hidden", "mean", "value", "dmean", "dvalue")


class ImInfo(C.Structure):
    _fields_ = [("n_bodies", C.c_int32), ("obs_dim", C.c_int32), ("action_dim", C.c_int32),
                ("n_clips", C.c_int32), ("n_layers", C.c_int32), ("policy_dtype", C.c_int32),
                ("max_depth", C.c_int32), ("max_envs", C.c_int64), ("device_bytes", C.c_int64)]


EXPORTED = ["im_create", "im_destroy", "im_get_info", "im_env_step_fused", "im_policy_act",
            "im_reset_envs", "im_standin_physics", "im_set_critic", "im_value",
            "im_policy_act_value", "im_gae", "im_gae_noalloc",
            "im_ppo_setup", "im_ppo_update", "im_ppo_grad", "im_ppo_params_get",
            "im_ppo_read", "im_status_str", "im_last_error"]
# measurement probes of the GPU (include/instantmimic_calib.h), not the method
CALIB_EXPORTED = ["im_calib_mfma", "im_calib_lds", "im_calib_read"]
IM_CALIB_MFMA_BF16, IM_CALIB_MFMA_F32 = 0, 1

_lib = None


def lib():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libinstantmimic.so is not built (run python -m "
                           "paper_2609_09821_amd.build); there is no fallback path")
    L = C.CDLL(LIB_PATH)
    st = C.c_int
    L.im_create.argtypes = [C.POINTER(ImConfig), C.POINTER(ImSkeleton), C.POINTER(ImClip),
                            C.c_int32, C.POINTER(ImPolicy), C.c_int64, C.POINTER(C.c_void_p)]
    L.im_create.restype = st
    L.im_destroy.argtypes = [C.c_void_p]
    L.im_destroy.restype = st
    L.im_get_info.argtypes = [C.c_void_p, C.POINTER(ImInfo)]
    L.im_get_info.restype = st
    L.im_env_step_fused.argtypes = [C.c_void_p, C.POINTER(ImEnvBufs), C.c_void_p]
    L.im_env_step_fused.restype = st
    L.im_policy_act.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p, C.c_int64,
                                C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    L.im_policy_act.restype = st
    L.im_reset_envs.argtypes = [C.c_void_p, C.POINTER(ImEnvBufs), C.c_void_p, C.c_void_p]
    L.im_reset_envs.restype = st
    L.im_standin_physics.argtypes = [C.c_void_p, C.POINTER(ImEnvBufs), C.c_float, C.c_float,
                                     C.c_void_p]
    L.im_standin_physics.restype = st
    L.im_set_critic.argtypes = [C.c_void_p, C.POINTER(ImPolicy)]
    L.im_set_critic.restype = st
    L.im_value.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_int64, C.c_void_p, C.c_void_p]
    L.im_value.restype = st
    L.im_policy_act_value.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p, C.c_int64,
                                      C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    L.im_policy_act_value.restype = st
    L.im_gae.argtypes = [C.c_void_p, C.POINTER(ImRollout), C.c_void_p]
    L.im_gae.restype = st
    L.im_gae_noalloc.argtypes = [C.POINTER(ImRollout), C.c_void_p]
    L.im_gae_noalloc.restype = st
    L.im_ppo_setup.argtypes = [C.c_void_p, C.c_int64]
    L.im_ppo_setup.restype = st
    L.im_ppo_update.argtypes = [C.c_void_p, C.POINTER(ImPpoBatch), C.POINTER(ImPpoParams), C.c_void_p]
    L.im_ppo_update.restype = st
    L.im_ppo_grad.argtypes = [C.c_void_p, C.POINTER(ImPpoBatch), C.POINTER(ImPpoParams), C.c_int32,
                              C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]
    L.im_ppo_grad.restype = st
    L.im_ppo_params_get.argtypes = [C.c_void_p, C.c_void_p, C.POINTER(C.c_int64), C.c_void_p]
    L.im_ppo_params_get.restype = st
    L.im_ppo_read.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.POINTER(C.c_int64),
                              C.POINTER(C.c_int64), C.POINTER(C.c_int64), C.c_void_p]
    L.im_ppo_read.restype = st
    L.im_status_str.argtypes = [C.c_int]
    L.im_status_str.restype = C.c_char_p
    L.im_last_error.argtypes = []
    L.im_last_error.restype = C.c_char_p
    L.im_calib_mfma.argtypes = [C.c_int, C.c_int64, C.c_int, C.c_void_p, C.c_void_p]
    L.im_calib_mfma.restype = st
    L.im_calib_lds.argtypes = [C.c_int, C.c_int, C.c_int64, C.c_int, C.c_void_p, C.c_void_p]
    L.im_calib_lds.restype = st
    L.im_calib_read.argtypes = [C.c_void_p, C.c_int64, C.c_int, C.c_int, C.c_void_p, C.c_void_p]
    L.im_calib_read.restype = st
    _lib = L
    return L


class ImError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s: %s" % (lib().im_status_str(status).decode(), msg))
        self.status = status


def _check(status):
    if status != IM_OK:
        raise ImError(status, lib().im_last_error().decode())


# ------------------------------------------------------------- C-named calls
def im_create(cfg, skel, clips, n_clips, policy, max_envs):
    out = C.c_void_p()
    _check(lib().im_create(C.byref(cfg), C.byref(skel), clips, n_clips, C.byref(policy),
                           int(max_envs), C.byref(out)))
    return out


def im_destroy(ctx):
    _check(lib().im_destroy(ctx))


def im_get_info(ctx):
    info = ImInfo()
    _check(lib().im_get_info(ctx, C.byref(info)))
    return info


def im_env_step_fused(ctx, bufs, stream=None):
    _check(lib().im_env_step_fused(ctx, C.byref(bufs), stream))


def im_policy_act(ctx, obs_ptr, ld_obs, env_n_ptr, n_envs, mean_ptr, action_ptr, logp_ptr,
                  stream=None):
    _check(lib().im_policy_act(ctx, obs_ptr, int(ld_obs), env_n_ptr, int(n_envs), mean_ptr,
                               action_ptr, logp_ptr, stream))


def im_reset_envs(ctx, bufs, mask_ptr=None, stream=None):
    _check(lib().im_reset_envs(ctx, C.byref(bufs), mask_ptr, stream))


def im_standin_physics(ctx, bufs, sigma_joint, sigma_vel, stream=None):
    _check(lib().im_standin_physics(ctx, C.byref(bufs), float(sigma_joint), float(sigma_vel),
                                    stream))


def im_set_critic(ctx, critic):
    _check(lib().im_set_critic(ctx, C.byref(critic)))


def im_value(ctx, obs_ptr, ld_obs, n_envs, value_ptr, stream=None):
    _check(lib().im_value(ctx, obs_ptr, int(ld_obs), int(n_envs), value_ptr, stream))


def im_policy_act_value(ctx, obs_ptr, ld_obs, env_n_ptr, n_envs, mean_ptr, action_ptr, logp_ptr,
                        value_ptr, stream=None):
    _check(lib().im_policy_act_value(ctx, obs_ptr, int(ld_obs), env_n_ptr, int(n_envs), mean_ptr,
                                     action_ptr, logp_ptr, value_ptr, stream))


def im_gae(ctx, rollout, stream=None):
    _check(lib().im_gae(ctx, C.byref(rollout), stream))


def im_gae_noalloc(rollout, stream=None):
    _check(lib().im_gae_noalloc(C.byref(rollout), stream))


def gae_noalloc(ro, gamma, lam, summary=True, stream=None):
    """im_gae_noalloc over a RolloutStorage (no context; the library's fixed
    scratch on the current device)."""
    im_gae_noalloc(ro.struct(gamma, lam, summary), _stream(stream))


def im_calib_mfma(kind, iters, blocks, out_ptr, stream=None):
    _check(lib().im_calib_mfma(int(kind), int(iters), int(blocks), out_ptr, stream))


def im_calib_lds(width, waves, iters, blocks, out_ptr, stream=None):
    _check(lib().im_calib_lds(int(width), int(waves), int(iters), int(blocks), out_ptr, stream))


def im_calib_read(src_ptr, nbytes, passes, blocks, out_ptr, stream=None):
    _check(lib().im_calib_read(src_ptr, int(nbytes), int(passes), int(blocks), out_ptr, stream))


def im_ppo_setup(ctx, max_minibatch):
    _check(lib().im_ppo_setup(ctx, int(max_minibatch)))


def im_ppo_update(ctx, batch, params, stream=None):
    _check(lib().im_ppo_update(ctx, C.byref(batch), C.byref(params), stream))


def im_ppo_grad(ctx, batch, params, epoch, minibatch, grad_ptr, stats_ptr, stream=None):
    _check(lib().im_ppo_grad(ctx, C.byref(batch), C.byref(params), int(epoch), int(minibatch),
                             grad_ptr, stats_ptr, stream))


def im_ppo_params_get(ctx, params_ptr=None, stream=None):
    n = C.c_int64()
    _check(lib().im_ppo_params_get(ctx, params_ptr, C.byref(n), stream))
    return n.value


def im_ppo_read(ctx, buffer, layer, dst_ptr=None, stream=None):
    r, c, e = C.c_int64(), C.c_int64(), C.c_int64()
    _check(lib().im_ppo_read(ctx, buffer, layer, dst_ptr, C.byref(r), C.byref(c), C.byref(e), stream))
    return r.value, c.value, e.value


# ------------------------------------------------------------- conveniences
def _f32(a):
    return np.ascontiguousarray(a, np.float32)


def _i32(a):
    return np.ascontiguousarray(a, np.int32)


def _ptr(a, ct):
    return a.ctypes.data_as(C.POINTER(ct))


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _dptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


class EnvBuffers:
    """Device buffers of a batch of envs (torch tensors) in the library layout."""

    def __init__(self, n_bodies, n_envs, ld=None, device="cuda", obs_dim=None, n_actions=0):
        import torch
        B = n_bodies
        ld = int(ld if ld is not None else n_envs)
        self.B, self.n_envs, self.ld = B, int(n_envs), ld
        f = dict(device=device, dtype=torch.float32)
        self.body_pos = torch.zeros((B, 3, ld), **f)
        self.body_quat = torch.zeros((B, 4, ld), **f)
        self.body_linvel = torch.zeros((B, 3, ld), **f)
        self.body_angvel = torch.zeros((B, 3, ld), **f)
        self.env_clip = torch.zeros(ld, device=device, dtype=torch.int32)
        self.env_phase = torch.zeros(ld, **f)
        self.env_t = torch.zeros(ld, device=device, dtype=torch.int32)
        self.env_n = torch.zeros(ld, device=device, dtype=torch.int32)  # uint32 bits
        self.reward = torch.zeros(ld, **f)
        self.terminated = torch.zeros(ld, device=device, dtype=torch.uint8)
        self.truncated = torch.zeros(ld, device=device, dtype=torch.uint8)
        self.obs = torch.zeros((15 * B + 1 if obs_dim is None else obs_dim, ld), **f)
        self.ref_frame = torch.zeros(ld, device=device, dtype=torch.int32)
        # the action applied in the step ([n_envs][A]), read when the observation
        # ends with the previous action
        self.prev_action = torch.zeros((max(self.n_envs, 1), n_actions), **f) if n_actions else None

    def struct(self, with_ref_frame=True):
        return ImEnvBufs(
            self.body_pos.data_ptr(), self.body_quat.data_ptr(), self.body_linvel.data_ptr(),
            self.body_angvel.data_ptr(), self.env_clip.data_ptr(), self.env_phase.data_ptr(),
            self.env_t.data_ptr(), self.env_n.data_ptr(), self.reward.data_ptr(),
            self.terminated.data_ptr(), self.truncated.data_ptr(), self.obs.data_ptr(),
            self.ref_frame.data_ptr() if with_ref_frame else None, self.n_envs, self.ld,
            None if self.prev_action is None else self.prev_action.data_ptr())

    SIM = ("body_pos", "body_quat", "body_linvel", "body_angvel")
    ENV = ("env_clip", "env_phase", "env_t", "env_n")


class Description:
    """The C structs of a synthetic world description (host memory only; the
    arrays they point to are kept alive by this object)."""

    def __init__(self, desc):
        sk = desc["skeleton"]
        cfg = desc["config"]
        pol = desc["policy"]
        keep = self._keep = []

        def k(a):
            keep.append(a)
            return a

        self.cfg = ImConfig(float(cfg["dt"]), float(cfg["h_term"]), float(cfg["r_min"]),
                            int(cfg["grace"]), float(cfg["c_pose"]), float(cfg["w_pos"]),
                            float(cfg["w_ee"]), float(cfg["c_vel"]), float(cfg["w_vel"]),
                            float(cfg["c_com"]), float(cfg["w_com"]), int(cfg["seed"]),
                            int(cfg.get("reward_form", 0)), float(cfg.get("m_jrot", 0.0)),
                            float(cfg.get("m_jvel", 0.0)), float(cfg.get("m_com", 0.0)),
                            float(cfg.get("m_eepos", 0.0)), float(cfg.get("m_eerot", 0.0)),
                            int(cfg.get("obs_future", 0)), int(cfg.get("obs_prev_action", 0)),
                            int(cfg.get("env_split", 0)))
        self.skel = ImSkeleton(int(sk["n_bodies"]), _ptr(k(_i32(sk["parent"])), C.c_int32),
                               _ptr(k(_i32(sk["jtype"])), C.c_int32),
                               _ptr(k(_f32(sk["axis"])), C.c_float),
                               _ptr(k(_f32(sk["offset"])), C.c_float),
                               _ptr(k(_f32(sk["mass"])), C.c_float))
        clips = desc["clips"]
        arr = (ImClip * len(clips))()
        for i, c in enumerate(clips):
            arr[i] = ImClip(int(c["n_frames"]), float(c["fps"]),
                            _ptr(k(_f32(c["root_pos"])), C.c_float),
                            _ptr(k(_f32(c["root_quat"])), C.c_float),
                            _ptr(k(_f32(c["local_quat"])), C.c_float))
        self.clips = arr
        self.n_clips = len(clips)
        self.policy = self._mlp(pol)
        self.critic = self._mlp(desc["critic"]) if desc.get("critic") is not None else None

    def _mlp(self, net):
        """ImPolicy of an MLP description (weights and biases kept alive here)."""
        keep = self._keep
        L = len(net["W"])
        dims = _i32(net["dims"])
        keep.append(dims)
        bf16 = bool(net["bf16"])
        wptrs = (C.c_void_p * L)()
        bptrs = (C.POINTER(C.c_float) * L)()
        for l in range(L):
            w = _f32(net["W"][l])
            if bf16:
                w = np.ascontiguousarray((w.view(np.uint32) >> 16).astype(np.uint16))
            keep.append(w)
            wptrs[l] = w.ctypes.data
            b = _f32(net["b"][l])
            keep.append(b)
            bptrs[l] = _ptr(b, C.c_float)
        keep += [wptrs, bptrs]
        log_std = net.get("log_std")
        ls = None
        if log_std is not None:
            ls = _f32(log_std)
            keep.append(ls)
        return ImPolicy(L, _ptr(dims, C.c_int32), IM_DTYPE_BF16 if bf16 else IM_DTYPE_F32,
                        wptrs, bptrs, None if ls is None else _ptr(ls, C.c_float))

    def create_status(self, max_envs):
        """Raw im_create: (status, context pointer or None)."""
        out = C.c_void_p()
        st = lib().im_create(C.byref(self.cfg), C.byref(self.skel), self.clips, self.n_clips,
                             C.byref(self.policy), int(max_envs), C.byref(out))
        return st, out


class Context:
    """A library context built from a synthetic world description."""

    def __init__(self, desc, max_envs, critic=True):
        d = self.desc = Description(desc)
        self.ptr = im_create(d.cfg, d.skel, d.clips, d.n_clips, d.policy, max_envs)
        if critic and d.critic is not None:
            im_set_critic(self.ptr, d.critic)
        self.info = im_get_info(self.ptr)

    def close(self):
        if getattr(self, "ptr", None):
            im_destroy(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- calls on tensors
    def buffers(self, n_envs, ld=None):
        prev = int(self.desc.cfg.obs_prev_action) != 0
        return EnvBuffers(self.info.n_bodies, n_envs, ld, obs_dim=self.info.obs_dim,
                          n_actions=self.info.action_dim if prev else 0)

    def env_step_fused(self, bufs, stream=None, with_ref_frame=True):
        im_env_step_fused(self.ptr, bufs.struct(with_ref_frame), _stream(stream))

    def reset_envs(self, bufs, mask=None, stream=None):
        im_reset_envs(self.ptr, bufs.struct(), _dptr(mask), _stream(stream))

    def standin_physics(self, bufs, sigma_joint, sigma_vel, stream=None):
        im_standin_physics(self.ptr, bufs.struct(), sigma_joint, sigma_vel, _stream(stream))

    def policy_act(self, obs, env_n, n_envs, mean, action, logp=None, stream=None):
        im_policy_act(self.ptr, _dptr(obs), obs.shape[1], _dptr(env_n), n_envs, _dptr(mean),
                      _dptr(action), _dptr(logp), _stream(stream))

    def value(self, obs, n_envs, value, stream=None):
        im_value(self.ptr, _dptr(obs), obs.shape[1], n_envs, _dptr(value), _stream(stream))

    def policy_act_value(self, obs, env_n, n_envs, mean, action, logp, value, stream=None):
        im_policy_act_value(self.ptr, _dptr(obs), obs.shape[1], _dptr(env_n), n_envs, _dptr(mean),
                            _dptr(action), _dptr(logp), _dptr(value), _stream(stream))

    def ppo_setup(self, max_minibatch):
        im_ppo_setup(self.ptr, max_minibatch)

    def ppo_update(self, batch, params, stream=None):
        im_ppo_update(self.ptr, batch, params, _stream(stream))

    def ppo_grad(self, batch, params, epoch, minibatch, grad, stats=None, stream=None):
        im_ppo_grad(self.ptr, batch, params, epoch, minibatch, _dptr(grad), _dptr(stats),
                    _stream(stream))

    def ppo_params(self, out=None, stream=None):
        """Number of parameters, or the master weights copied into `out`."""
        if out is None:
            return im_ppo_params_get(self.ptr)
        return im_ppo_params_get(self.ptr, _dptr(out), _stream(stream))

    def ppo_read(self, name, layer=0, stream=None):
        """A copy (device tensor [rows][cols]) of the update buffer `name`
        (PPO_BUFFERS) of the last minibatch; bf16 buffers as torch.bfloat16."""
        import torch
        k = PPO_BUFFERS.index(name)
        rows, cols, eb = im_ppo_read(self.ptr, k, layer)
        out = torch.empty((rows, cols), dtype=torch.bfloat16 if eb == 2 else torch.float32,
                          device="cuda")
        im_ppo_read(self.ptr, k, layer, _dptr(out), _stream(stream))
        return out

    def gae(self, ro, gamma, lam, summary=True, stream=None):
        """GAE (and, with summary, the rollout summaries) over a RolloutStorage."""
        im_gae(self.ptr, ro.struct(gamma, lam, summary), _stream(stream))


class RolloutStorage:
    """Device storage of a T-step rollout, written in place by the step calls:
    step t's policy and value read obs[t] and write action/mean/logp/value
    slot t; the fused env step writes reward/terminated/truncated slot t and
    obs[t + 1].  `env_bufs(t)` points an EnvBuffers at those slots."""

    def __init__(self, ctx, n_envs, T, ld=None, device="cuda"):
        import torch
        ld = int(ld if ld is not None else n_envs)
        D, A = ctx.info.obs_dim, ctx.info.action_dim
        self.T, self.n_envs, self.ld = int(T), int(n_envs), ld
        f = dict(device=device, dtype=torch.float32)
        u8 = dict(device=device, dtype=torch.uint8)
        self.obs = torch.zeros((T + 1, D, ld), **f)
        self.mean = torch.zeros((T, max(n_envs, 1), A), **f)
        self.action = torch.zeros((T, max(n_envs, 1), A), **f)
        self.logp = torch.zeros((T, ld), **f)
        self.value = torch.zeros((T + 1, ld), **f)
        self.reward = torch.zeros((T, ld), **f)
        self.terminated = torch.zeros((T, ld), **u8)
        self.truncated = torch.zeros((T, ld), **u8)
        self.advantage = torch.zeros((T, ld), **f)
        self.ret = torch.zeros((T, ld), **f)
        self.ep_return = torch.zeros(ld, **f)
        self.ep_length = torch.zeros(ld, device=device, dtype=torch.int32)
        self.summary = torch.zeros(len(SUMMARY_FIELDS), device=device, dtype=torch.float64)

    def env_bufs(self, bufs, t):
        """`bufs` (sim and env state) with its step outputs pointed at slot t."""
        assert bufs.ld == self.ld and bufs.n_envs == self.n_envs
        bufs.reward = self.reward[t]
        bufs.terminated = self.terminated[t]
        bufs.truncated = self.truncated[t]
        bufs.obs = self.obs[t + 1]
        if bufs.prev_action is not None:
            bufs.prev_action = self.action[t]
        return bufs

    def struct(self, gamma, lam, summary=True):
        return ImRollout(self.T, self.n_envs, self.ld, float(gamma), float(lam),
                         self.reward.data_ptr(), self.terminated.data_ptr(),
                         self.truncated.data_ptr(), self.value.data_ptr(),
                         self.advantage.data_ptr(), self.ret.data_ptr(),
                         self.ep_return.data_ptr(), self.ep_length.data_ptr(),
                         self.summary.data_ptr() if summary else None)


# PPO defaults: the baseline column of the backflip configuration table (ratio
# clip, value and entropy coefficients, KL threshold, learning epochs) and the
# usual Adam / norm-clip settings
PPO_DEFAULTS = dict(clip=0.2, value_coef=2.0, entropy_coef=0.0, clipped_value_loss=1,
                    max_grad_norm=1.0, beta1=0.9, beta2=0.999, eps=1e-8, desired_kl=0.008,
                    lr_min=1e-5, lr_max=1e-2, epochs=5, minibatches=4)


def ppo_params(**over):
    p = dict(PPO_DEFAULTS, **over)
    return ImPpoParams(*(p[k] for k, _ in ImPpoParams._fields_))


def ppo_batch(ro, perm, lr, stats=None):
    """ImPpoBatch over a RolloutStorage after im_gae; perm: device int32
    [epochs][T * n_envs / 64]; lr: device float [1]; stats: device float64
    [len(PPO_STATS)] or None."""
    return ImPpoBatch(ro.T, ro.n_envs, ro.ld, ro.obs.data_ptr(), ro.action.data_ptr(),
                      ro.mean.data_ptr(), ro.logp.data_ptr(), ro.value.data_ptr(),
                      ro.advantage.data_ptr(), ro.ret.data_ptr(), ro.summary.data_ptr(),
                      perm.data_ptr(), lr.data_ptr(), None if stats is None else stats.data_ptr())
