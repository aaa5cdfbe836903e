"""Oracle of the rollout-end computations: generalized advantage estimation
and the rollout summaries.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's training loop (Fig. 3) writes (obs, action, reward, terminated,
truncated) to the rollout storage at every step and hands the storage to the
PPO update; its configuration table (Appendix) lists the discount factor
gamma and the GAE parameter lambda.  GAE itself is Schulman et al.'s
(High-Dimensional Continuous Control Using Generalized Advantage Estimation,
2016): the advantage is the (gamma lambda)-discounted sum of the one-step TD
errors delta_t = r_t + gamma V(s_{t+1}) - V(s_t) up to the end of the episode.
Readings taken here (the paper is silent on them):
  * an env that terminates at step t has no successor: delta_t = r_t - V_t
    and the sum stops at t;
  * an env truncated at t (phase end, not terminated) is cut off, not failed:
    its successor's value is bootstrapped, and since the observation after
    the step is already the reset one, V_t (the value of the observation the
    action was taken on) stands in for it: delta_t = r_t + gamma V_t - V_t;
    the sum also stops at t;
  * past the last step of the rollout the sum stops, and V_T (the value of
    the observation after the last step) bootstraps delta_{T-1};
  * returns R_t = A_t + V_t.
Here the advantage is written as the sum itself, term by term, in float64
(the GPU evaluates the equivalent backward recursion).
"""
import numpy as np

SUMMARY_FIELDS = ("reward_sum", "n_terminated", "n_truncated", "n_episodes",
                  "episode_return_sum", "episode_length_sum", "advantage_sum",
                  "advantage_sq_sum", "value_sum", "return_sum")


def _delta(reward, term, trunc, value, gamma):
    """One-step TD errors [T][N] (float64) with the readings above."""
    T = reward.shape[0]
    r = reward.astype(np.float64)
    V = value.astype(np.float64)
    te = term.astype(bool)
    tr = trunc.astype(bool) & ~te
    nxt = np.where(te, 0.0, np.where(tr, V[:T], V[1:T + 1]))
    return r + gamma * nxt - V[:T]


def gae(reward, term, trunc, value, gamma, lam):
    """reward, term, trunc: [T][N]; value: [T+1][N].  Returns (advantage,
    return) [T][N] float32, the sums written out."""
    reward = np.asarray(reward)
    T, N = reward.shape
    delta = _delta(reward, np.asarray(term), np.asarray(trunc), np.asarray(value), gamma)
    done = np.asarray(term).astype(bool) | np.asarray(trunc).astype(bool)
    adv = np.zeros((T, N), np.float64)
    for t in range(T):
        alive = np.ones(N, bool)          # the sum still runs for this env
        acc = np.zeros(N, np.float64)
        w = 1.0
        for u in range(t, T):
            acc += np.where(alive, w * delta[u], 0.0)
            alive &= ~done[u]             # the episode ends at u
            w *= gamma * lam
        adv[t] = acc
    ret = adv + np.asarray(value)[:T].astype(np.float64)
    return adv.astype(np.float32), ret.astype(np.float32)


def rollout_summary(reward, term, trunc, value, adv, ret, ep_return, ep_length):
    """Rollout summaries (float64 [10], fields SUMMARY_FIELDS) and the updated
    running-episode accumulators.

    ep_return [N] float32 / ep_length [N] int32: return and length of the
    episode each env is in, carried across rollouts.  At every step the
    reward is added to the return (float32, step order) and the length grows
    by one; an env that is terminated or truncated closes its episode (its
    return and length enter the sums) and starts the next one at 0.
    Advantage, value and return sums are over the stored float32 values."""
    reward = np.asarray(reward, np.float32)
    T, N = reward.shape
    term = np.asarray(term).astype(bool)
    trunc = np.asarray(trunc).astype(bool)
    epr = np.array(ep_return, np.float32, copy=True)
    epl = np.array(ep_length, np.int64, copy=True)
    s = dict.fromkeys(SUMMARY_FIELDS, 0.0)
    for t in range(T):
        for e in range(N):
            r = reward[t, e]
            s["reward_sum"] += float(r)
            epr[e] = np.float32(epr[e] + r)
            epl[e] += 1
            if term[t, e]:
                s["n_terminated"] += 1
            if trunc[t, e]:
                s["n_truncated"] += 1
            if term[t, e] or trunc[t, e]:
                s["n_episodes"] += 1
                s["episode_return_sum"] += float(epr[e])
                s["episode_length_sum"] += float(epl[e])
                epr[e] = 0.0
                epl[e] = 0
            a = float(adv[t, e])
            s["advantage_sum"] += a
            s["advantage_sq_sum"] += a * a
            s["value_sum"] += float(value[t, e])
            s["return_sum"] += float(ret[t, e])
    out = np.array([s[k] for k in SUMMARY_FIELDS], np.float64)
    return out, epr, epl.astype(np.int32)
