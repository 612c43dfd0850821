"""Token-level truncated importance sampling (TIS) weights and the mismatch KL --
oracle, test infrastructure only.

Section 2.1.3: rollouts come from the FP8 policy while training assumes the bf16
policy, so each sampled token is reweighted by w = pi_theta / pi_theta^FP8
(Eq. (2)), evaluated at token level from the two policies' log-probabilities of
the sampled token, and the weight is truncated at C (Eq. (3); C = 2 throughout
the paper).  Section 2.2 tracks the mismatch KL D_KL(pi^FP8 || pi_theta) over the
same tokens.  Readings taken here (listed with their reasons in the project's
design notes):

  * w = exp(logp_train - logp_rollout), computed from the fp32 inputs in fp64;
    w_TIS = min(w, C) (truncation from above; w > 0 already), rounded once to
    fp32; tokens outside the response mask get w_TIS = 0;
  * the mismatch KL is estimated from the sampled tokens (drawn from pi^FP8) with
    the per-token terms k1 = logp_rollout - logp_train (the definition's
    Monte-Carlo form) and k3 = (w - 1) - log w = expm1(d) - d, d = logp_train -
    logp_rollout (non-negative, same expectation); the outputs are their sums
    over valid tokens, the valid-token count and the number of truncated tokens,
    all in fp64.
"""
import numpy as np


def tis_weights_kl(logp_train, logp_rollout, mask=None, clip_c: float = 2.0):
    """Returns (w_tis fp32 [n], stats fp64 [4] = (sum k1, sum k3, valid count, truncated count))."""
    lt = np.asarray(logp_train, dtype=np.float32).astype(np.float64)
    lr = np.asarray(logp_rollout, dtype=np.float32).astype(np.float64)
    valid = np.ones(lt.shape, bool) if mask is None else np.asarray(mask).astype(bool)
    d = lt - lr                                          # exact: both fp32
    with np.errstate(over="ignore"):
        w = np.exp(d)
        k3 = np.expm1(d) - d
    c = float(np.float32(clip_c))
    w_tis = np.where(valid, np.minimum(w, c), 0.0).astype(np.float32)
    stats = np.array([np.sum(np.where(valid, -d, 0.0)), np.sum(np.where(valid, k3, 0.0)),
                      float(valid.sum()), float((valid & (w > c)).sum())], dtype=np.float64)
    return w_tis, stats
