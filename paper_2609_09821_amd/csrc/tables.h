// tables.h -- device-resident tables owned by a context and the argument
// blocks of the env kernels.
#pragma once

#include <stdint.h>

#include "../../include/instantmimic.h"

namespace im {

// Most root-to-leaf walks of the path-split fused step.
constexpr int IM_MAX_PATHS = 8;

// Skeleton, reordered into depth-first preorder: a body's parent is then
// either the previous body or a branch point whose frame was parked.  Read
// with wave-uniform loads.
struct SkelTab {
    int32_t B;          // bodies
    int32_t n_slots;    // parked-frame slots needed (nested branch points)
    int32_t n_dof;      // rotational DoFs of the joints (stand-in noise)
    int32_t body[IM_MAX_BODIES];   // body index at preorder position i
    int32_t depth[IM_MAX_BODIES];  // its depth (root 0)
    int32_t bslot[IM_MAX_BODIES];  // LDS slot of its frame if it has >= 2 children, else -1
    int32_t pslot[IM_MAX_BODIES];  // slot of its parent if the parent is not the
                                   // previous body in preorder, else -1
    int32_t jtype[IM_MAX_BODIES];
    int32_t leaf[IM_MAX_BODIES];
    int32_t zrot[IM_MAX_BODIES];   // first stand-in normal of its rotation noise
    float offset[IM_MAX_BODIES][4];
    float axis[IM_MAX_BODIES][4];
    float massw[IM_MAX_BODIES];    // m_b / sum m
    int32_t pbody[IM_MAX_BODIES];  // by body index: its parent (-1 for the root)
    int32_t ee_slot[IM_MAX_BODIES];  // observation slot of the future frames: 0 the
                                     // root, 1.. the end effectors in body order, -1 none
    int32_t n_ee;                  // end effectors (leaves)
    // The fused step for small batches runs every env on several threads, each
    // walking the bodies it owns plus their ancestors (a PartWalk): either two
    // halves, or one walk per root-to-leaf path of the skeleton.
    struct PartWalk {
        int32_t n;                     // positions of the walk (root first, preorder)
        int32_t body[IM_MAX_BODIES];   // body at position i
        int32_t rec[IM_MAX_BODIES];    // its position in the full preorder (segment record)
        int32_t own[IM_MAX_BODIES];    // 1: errors, reset and observation of this body
                                       // belong to this walk; 0: an ancestor passed through
        int32_t bslot[IM_MAX_BODIES];  // as above, for the walk's own branch points
        int32_t pslot[IM_MAX_BODIES];
        int32_t jtype[IM_MAX_BODIES];
        int32_t leaf[IM_MAX_BODIES];   // leaf of the whole skeleton (end effector)
        float offset[IM_MAX_BODIES][4];
        float massw[IM_MAX_BODIES];
        int32_t n_own;                 // bodies this walk owns, in walk order
        int32_t own_body[IM_MAX_BODIES];
    };
    int32_t half_slots;            // parked-frame slots needed by either half walk
    PartWalk half[2];
    // Path walks: path p runs from the root to the p-th leaf in preorder and owns
    // the bodies on it that no earlier path owns.  n_paths = 0 when the skeleton
    // has more than IM_MAX_PATHS leaves.
    int32_t n_paths;
    int32_t path_slots;            // 0: a path has no branch point
    PartWalk path[IM_MAX_PATHS];
};

// Per clip.  seg_base: float4 index of segment 0 in the segment table.
struct ClipTab {
    int32_t F;
    float dphi;   // float(dt * fps / (F - 1))
    float fm1;    // float(F - 1)
    int32_t seg_base;
};

// Segment table: for every clip k and segment i0 in [0, F-2], a record of
// 6 + 3 (B - 1) float4 in preorder:
//   root   [0] = (A.x, A.y, A.z, d.x)     anchor A = root position of frame i0
//          [1] = (d.y, d.z, v.x, v.y)     d = P(i0+1) - P(i0), v = d * fps
//          [2] = (v.z, w.x, w.y, w.z)     w = rotvec(Q1 Q0^-1) * fps (world)
//          [3] = a                        slerp basis: q(alpha) = cos(alpha W) a
//          [4] = u                                           + sin(alpha W) u
//          [5] = (W, 0, 0, 0)
//   joint  [0] = a, [1] = u, [2] = (w.x, w.y, w.z, W)  (w in the parent frame)
// a = q0/|q0|, b = +-q1/|q1| on a's hemisphere, W = angle between a and b,
// u = unit component of b orthogonal to a.
__host__ __device__ inline int seg_stride(int B) { return 6 + 3 * (B - 1); }

struct EnvArgs {
    const SkelTab *sk;
    const ClipTab *clips;
    const float4 *seg;
    float *pos, *quat, *linvel, *angvel;
    int32_t *env_clip;
    float *env_phase;
    int32_t *env_t;
    uint32_t *env_n;
    float *reward;
    uint8_t *term, *trunc;
    float *obs;
    int32_t *ref_frame;
    const uint8_t *mask;
    int64_t n, ld;
    uint64_t seed;
    int32_t n_clips;
    int32_t grace;
    float h_term, r_min;
    float c_pose, w_pos, w_ee, c_vel, w_vel, c_com, w_com;
    float sigma_joint, sigma_vel;
    // training terms
    int32_t reward_form;       // IM_REWARD_GROUPED or IM_REWARD_MULTIPLICATIVE
    int32_t obs_prev;          // previous-action rows in the observation
    float m_jrot, m_jvel, m_com, m_eepos, m_eerot;
    int32_t obs_future;        // future reference frames in the observation
    int32_t obs_base;          // first observation row after the phase (15 B + 1)
    int32_t A;                 // action width (previous-action rows)
    const float *prev_action;  // [n][A] (read by the step when obs_prev)
    // split fused step: its walks and their count (threads per env)
    const SkelTab::PartWalk *walks;
    int32_t n_parts;
};

}  // namespace im
