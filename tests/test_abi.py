"""The C ABI without a GPU: the library loads, exports every function the
header declares, and rejects malformed descriptions and calls with the
documented status codes before it touches the device."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2609_09821_amd import binding, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "instantmimic.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        from paper_2609_09821_amd import build
        build.build()
    return binding.lib()


CALIB_HEADER = os.path.join(ROOT, "include", "instantmimic_calib.h")


def _declared(path=HEADER):
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return sorted(set(re.findall(r"\b(im_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("im_create", "im_destroy", "im_env_step_fused", "im_policy_act", "im_reset_envs",
              "im_status_str", "im_last_error"):
        assert n in names
    assert sorted(binding.EXPORTED) == names


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    missing = [n for n in _declared() if n not in exported]
    assert not missing, missing
    for n in _declared():
        assert getattr(lib, n) is not None
    # C linkage: no mangled im_ entry points
    assert not [s for s in exported if s.startswith("_Z") and "im_" in s and "im::" not in s
                and re.match(r"_Z\d+im_", s)]


def test_status_strings(lib):
    names = ["IM_OK", "IM_ERR_INVALID_ARG", "IM_ERR_UNSUPPORTED", "IM_ERR_OOM", "IM_ERR_HIP"]
    for code, name in enumerate(names):
        assert lib.im_status_str(code).decode() == name
    assert lib.im_status_str(99).decode() == "unknown im_status"
    hdr = open(HEADER).read()
    for code, name in enumerate(names):
        assert re.search(r"\b%s\s*=\s*%d\b" % (name, code), hdr), name


def _status(desc, max_envs=64):
    d = binding.Description(desc)
    return d, d.create_status(max_envs)


def _expect(lib, st, code, words):
    assert st == code, (lib.im_status_str(st).decode(), lib.im_last_error().decode())
    msg = lib.im_last_error().decode()
    assert words in msg, msg


def _world(cfg=2, **over):
    return synth.make_world(cfg, n_envs=64, **over)


def test_create_rejects_null_pointers(lib):
    d = binding.Description(_world())
    out = C.c_void_p()
    st = lib.im_create(None, C.byref(d.skel), d.clips, d.n_clips, C.byref(d.policy), 64, C.byref(out))
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "NULL description")
    st = lib.im_create(C.byref(d.cfg), C.byref(d.skel), d.clips, d.n_clips, C.byref(d.policy), 64, None)
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "NULL out")
    assert out.value is None


@pytest.mark.parametrize("field,value,code,words", [
    ("dt", 0.0, binding.IM_ERR_INVALID_ARG, "dt"),
    ("dt", float("nan"), binding.IM_ERR_INVALID_ARG, "dt"),
    ("h_term", float("inf"), binding.IM_ERR_INVALID_ARG, "thresholds"),
    ("r_min", float("nan"), binding.IM_ERR_INVALID_ARG, "thresholds"),
    ("grace", -1, binding.IM_ERR_INVALID_ARG, "grace"),
    ("w_ee", float("nan"), binding.IM_ERR_INVALID_ARG, "weights"),
    ("reward_form", 2, binding.IM_ERR_INVALID_ARG, "reward_form"),
    ("m_jvel", float("inf"), binding.IM_ERR_INVALID_ARG, "multiplicative"),
    ("obs_future", 5, binding.IM_ERR_INVALID_ARG, "obs_future"),
    ("obs_prev_action", 3, binding.IM_ERR_INVALID_ARG, "obs_prev_action"),
    ("env_split", 4, binding.IM_ERR_INVALID_ARG, "env_split"),
    ("env_split", -1, binding.IM_ERR_INVALID_ARG, "env_split"),
])
def test_create_rejects_bad_config(lib, field, value, code, words):
    d = binding.Description(_world())
    setattr(d.cfg, field, value)
    st, out = d.create_status(64)
    _expect(lib, st, code, words)
    assert out.value is None


def test_create_rejects_bad_skeletons(lib):
    w = _world()
    sk = w["skeleton"]
    cases = []
    p = sk["parent"].copy(); p[5] = 7
    cases.append(("parent", p, "parent[b]"))
    p = sk["parent"].copy(); p[0] = 0
    cases.append(("parent", p, "parent[0]"))
    j = sk["jtype"].copy(); j[0] = binding.IM_JOINT_SPHERICAL
    cases.append(("jtype", j, "free joint"))
    j = sk["jtype"].copy(); j[3] = 17
    cases.append(("jtype", j, "joint type"))
    m = sk["mass"].copy(); m[2] = 0.0
    cases.append(("mass", m, "masses"))
    o = sk["offset"].copy(); o[4, 1] = np.inf
    cases.append(("offset", o, "finite"))
    for key, val, words in cases:
        w2 = dict(w, skeleton=dict(sk, **{key: val}))
        _, (st, out) = _status(w2)
        _expect(lib, st, binding.IM_ERR_INVALID_ARG, words)


def test_create_path_split_needs_at_most_eight_leaves(lib):
    # every body a child of the root: 14 leaves, more than the path split takes
    w = _world()
    sk = w["skeleton"]
    star = dict(w, skeleton=dict(sk, parent=np.where(np.arange(sk["n_bodies"]) == 0, -1, 0)
                                 .astype(np.int32)))
    star["config"] = dict(w["config"], env_split=binding.IM_SPLIT_PATHS)
    _, (st, out) = _status(star)
    _expect(lib, st, binding.IM_ERR_UNSUPPORTED, "leaves")
    assert out.value is None


def test_create_rejects_non_unit_revolute_axis(lib):
    w = _world()
    sk = w["skeleton"]
    rev = [b for b in range(1, sk["n_bodies"]) if sk["jtype"][b] == binding.IM_JOINT_REVOLUTE]
    assert rev
    ax = sk["axis"].copy()
    ax[rev[0]] *= 1.01
    _, (st, _) = _status(dict(w, skeleton=dict(sk, axis=ax)))
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "revolute axis")


def test_create_rejects_bad_clips(lib):
    w = _world()
    c0 = w["clips"][0]
    bad = []
    bad.append((dict(c0, n_frames=1, root_pos=c0["root_pos"][:1], root_quat=c0["root_quat"][:1],
                     local_quat=c0["local_quat"][:1]), "n_frames"))
    bad.append((dict(c0, fps=0.0), "fps"))
    q = c0["root_quat"].copy(); q[3] *= 1.01
    bad.append((dict(c0, root_quat=q), "root quaternion"))
    lq = c0["local_quat"].copy(); lq[2, 0] *= 1.01
    bad.append((dict(c0, local_quat=lq), "quaternion"))
    rp = c0["root_pos"].copy(); rp[1, 2] = np.nan
    bad.append((dict(c0, root_pos=rp), "finite"))
    for clip, words in bad:
        _, (st, _) = _status(dict(w, clips=[clip]))
        _expect(lib, st, binding.IM_ERR_INVALID_ARG, words)
    _, (st, _) = _status(dict(w, clips=[]))
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "n_clips")


def test_create_rejects_fixed_joint_rotation(lib):
    w = _world()
    sk = w["skeleton"]
    fixed = [b for b in range(1, sk["n_bodies"]) if sk["jtype"][b] == binding.IM_JOINT_FIXED]
    assert fixed
    c0 = w["clips"][0]
    lq = c0["local_quat"].copy()
    lq[0, fixed[0] - 1] = np.array([np.cos(0.2), np.sin(0.2), 0.0, 0.0], np.float32)
    _, (st, _) = _status(dict(w, clips=[dict(c0, local_quat=lq)]))
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "fixed joint")


def test_create_rejects_bad_policies(lib):
    w = _world()
    pol = w["policy"]
    dims = list(pol["dims"])
    bad_in = dict(pol, dims=[dims[0] + 1] + dims[1:])
    _, (st, _) = _status(dict(w, policy=bad_in))
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "observation width")
    ls = pol["log_std"].copy(); ls[0] = np.nan
    _, (st, _) = _status(dict(w, policy=dict(pol, log_std=ls)))
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "log_std")
    d = binding.Description(w)
    d.policy.dtype = 7
    st, _ = d.create_status(64)
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "dtype")
    d = binding.Description(w)
    d.policy.weight[1] = None
    st, _ = d.create_status(64)
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "NULL weight")


def test_create_checks_the_observation_width_of_the_training_terms(lib):
    # 2 future frames and the previous action widen the observation: a policy
    # sized for 15 B + 1 is rejected, one sized for D = 538 passes validation
    w = synth.make_world(6, n_envs=64)
    d = binding.Description(w)
    d.cfg.obs_future = 1
    st, _ = d.create_status(64)
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "observation width 484")
    d = binding.Description(w)
    d.cfg.obs_prev_action = 0
    st, _ = d.create_status(64)
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "observation width 469")


def test_create_reports_unsupported_sizes(lib):
    w = _world()
    pol = w["policy"]
    big = dict(pol, dims=list(pol["dims"][:-1]) + [129],
               W=pol["W"][:-1] + [np.zeros((129, pol["dims"][-2]), np.float32)],
               b=pol["b"][:-1] + [np.zeros(129, np.float32)], log_std=np.zeros(129, np.float32))
    _, (st, _) = _status(dict(w, policy=big))
    _expect(lib, st, binding.IM_ERR_UNSUPPORTED, "action width")
    d = binding.Description(w)
    d.skel.n_bodies = 65
    st, _ = d.create_status(64)
    _expect(lib, st, binding.IM_ERR_UNSUPPORTED, "IM_MAX_BODIES")


@pytest.mark.parametrize("max_envs", [0, -5, 1 << 32])
def test_create_rejects_bad_max_envs(lib, max_envs):
    _, (st, _) = _status(_world(), max_envs)
    _expect(lib, st, binding.IM_ERR_INVALID_ARG, "max_envs")


def test_calls_reject_null_context(lib):
    bufs = binding.ImEnvBufs()
    _expect(lib, lib.im_env_step_fused(None, C.byref(bufs), None), binding.IM_ERR_INVALID_ARG, "NULL context")
    _expect(lib, lib.im_reset_envs(None, C.byref(bufs), None, None), binding.IM_ERR_INVALID_ARG, "NULL context")
    _expect(lib, lib.im_standin_physics(None, C.byref(bufs), 0.1, 0.1, None), binding.IM_ERR_INVALID_ARG,
            "NULL context")
    _expect(lib, lib.im_policy_act(None, None, 1, None, 1, None, None, None, None),
            binding.IM_ERR_INVALID_ARG, "NULL context")
    _expect(lib, lib.im_destroy(None), binding.IM_ERR_INVALID_ARG, "NULL context")
    d = binding.Description(_world())
    _expect(lib, lib.im_set_critic(None, C.byref(d.critic)), binding.IM_ERR_INVALID_ARG,
            "NULL context")
    _expect(lib, lib.im_value(None, None, 1, 1, None, None), binding.IM_ERR_INVALID_ARG,
            "NULL context")
    _expect(lib, lib.im_policy_act_value(None, None, 1, None, 1, None, None, None, None, None),
            binding.IM_ERR_INVALID_ARG, "NULL context")
    ro = binding.ImRollout()
    _expect(lib, lib.im_gae(None, C.byref(ro), None), binding.IM_ERR_INVALID_ARG, "NULL context")
    pb, pp = binding.ImPpoBatch(), binding.ppo_params()
    _expect(lib, lib.im_ppo_setup(None, 64), binding.IM_ERR_INVALID_ARG, "NULL context")
    _expect(lib, lib.im_ppo_update(None, C.byref(pb), C.byref(pp), None), binding.IM_ERR_INVALID_ARG,
            "NULL context")
    _expect(lib, lib.im_ppo_grad(None, C.byref(pb), C.byref(pp), 0, 0, None, None, None),
            binding.IM_ERR_INVALID_ARG, "NULL context")
    n = C.c_int64()
    _expect(lib, lib.im_ppo_params_get(None, None, C.byref(n), None), binding.IM_ERR_INVALID_ARG,
            "NULL context")
    info = binding.ImInfo()
    _expect(lib, lib.im_get_info(None, C.byref(info)), binding.IM_ERR_INVALID_ARG, "NULL")


def test_binding_raises_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        binding.lib()


def test_calibration_probes_exported_and_argument_checks(lib):
    # the measurement probes' header: every declared function is exported, and
    # bad arguments are refused before anything is launched (no GPU here)
    names = _declared(CALIB_HEADER)
    assert sorted(binding.CALIB_EXPORTED) == names
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    assert not [n for n in names if n not in exported]
    buf = C.c_void_p(256)
    bad = 1   # IM_ERR_INVALID_ARG
    assert lib.im_calib_mfma(2, 10, 1, buf, None) == bad
    assert lib.im_calib_mfma(binding.IM_CALIB_MFMA_BF16, 0, 1, buf, None) == bad
    assert lib.im_calib_mfma(binding.IM_CALIB_MFMA_F32, 10, 0, buf, None) == bad
    assert lib.im_calib_mfma(binding.IM_CALIB_MFMA_F32, 10, 1, None, None) == bad
    assert lib.im_calib_lds(12, 4, 10, 1, buf, None) == bad
    assert lib.im_calib_lds(16, 0, 10, 1, buf, None) == bad
    assert lib.im_calib_lds(16, 17, 10, 1, buf, None) == bad
    assert lib.im_calib_lds(8, 4, 0, 1, buf, None) == bad
    assert lib.im_calib_read(buf, 24, 1, 1, buf, None) == bad        # not a multiple of 16
    assert lib.im_calib_read(C.c_void_p(264), 32, 1, 1, buf, None) == bad   # unaligned
    assert lib.im_calib_read(None, 32, 1, 1, buf, None) == bad
    assert lib.im_calib_read(buf, 32, 0, 1, buf, None) == bad
