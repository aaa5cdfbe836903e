"""Small hand-made worlds for tests (same dict format as synth.make_world)."""
import numpy as np

from paper_2609_09821_amd import synth


def custom_world(parent, jtype, offset, mass, clips, axis=None, **cfg_over):
    B = len(parent)
    skel = dict(
        name="custom", n_bodies=B, names=["b%d" % i for i in range(B)],
        parent=np.asarray(parent, np.int32), jtype=np.asarray(jtype, np.int32),
        axis=np.asarray(axis if axis is not None else np.zeros((B, 3)), np.float32),
        offset=np.asarray(offset, np.float32), mass=np.asarray(mass, np.float32),
    )
    pol = synth.make_policy(np.random.default_rng(0), [15 * B + 1, 8, 4], False)
    return dict(id=0, spec={}, n_envs=1, skeleton=skel, clips=clips, policy=pol,
                config=synth.step_config(0, **cfg_over), sigma_joint=0.05, sigma_vel=0.5)


def clip_from_arrays(root_pos, root_quat, local_quat, fps=30.0):
    root_pos = np.asarray(root_pos, np.float32)
    return dict(n_frames=root_pos.shape[0], fps=float(fps), root_pos=root_pos,
                root_quat=np.asarray(root_quat, np.float32),
                local_quat=np.asarray(local_quat, np.float32))


def rest_offsets_world(world_desc):
    """Root-to-body sum of rest offsets for every body (identity pose)."""
    sk = world_desc["skeleton"]
    B = sk["n_bodies"]
    P = np.zeros((B, 3))
    for b in range(1, B):
        P[b] = P[sk["parent"][b]] + sk["offset"][b].astype(np.float64)
    return P
