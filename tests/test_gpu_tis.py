"""GPU parity of the token-level TIS weights and mismatch-KL sums (section 2.1.3,
Eq. (2)-(3)) against the CPU oracle.  Both sides evaluate e^d in fp64 and round
min(e^d, C) once to fp32, so the weights may differ only where two fp64 exp
implementations round differently across an fp32 rounding boundary (at most one
fp32 ulp, expected nowhere); counts are exact; the fp64 sums agree to 1e-12 of the
sum of the terms' magnitudes (summation order differs)."""
import numpy as np
import pytest
import torch

import synth
from oracle import tis
from tests.gpu_util import announce, need_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fp8rl():
    need_gpu()
    import paper_2601_18150_amd as m
    m.load()
    return m


def check_tis(w_gpu, s_gpu, lt, lr, mask, c):
    w_ref, s_ref = tis.tis_weights_kl(lt, lr, mask, c)
    w = w_gpu.cpu().numpy()
    s = s_gpu.cpu().numpy()
    ulp = np.abs(w.view(np.int32).astype(np.int64) - w_ref.view(np.int32).astype(np.int64))
    assert ulp.max(initial=0) <= 1, f"weights differ by {ulp.max()} ulp"
    assert (ulp != 0).sum() <= max(1, w.size // 10**6), f"{(ulp != 0).sum()} weights differ"
    d = lt.astype(np.float64) - lr.astype(np.float64)
    valid = np.ones(d.shape, bool) if mask is None else mask.astype(bool)
    mag1 = np.abs(d[valid]).sum()
    mag3 = np.abs(np.expm1(d[valid]) - d[valid]).sum()
    assert abs(s[0] - s_ref[0]) <= 1e-12 * mag1 + 1e-300, (s[0], s_ref[0])
    assert abs(s[1] - s_ref[1]) <= 1e-12 * mag3 + 1e-300, (s[1], s_ref[1])
    assert s[2] == s_ref[2] and abs(s[3] - s_ref[3]) <= (ulp != 0).sum(), (s, s_ref)
    return w_ref, s_ref


@pytest.mark.parametrize("n,masked", [(0, False), (1, True), (255, False), (257, True), (1000, True),
                                      (300001, False)])
def test_tis_ragged_sizes(fp8rl, n, masked):
    announce(f"tis n={n} masked={masked}")
    rng = np.random.default_rng(n + 7)
    lr = -rng.exponential(0.4, n).astype(np.float32)
    lt = (lr + rng.normal(0, 0.3, n)).astype(np.float32)
    mask = (rng.uniform(0, 1, n) < 0.8).astype(np.uint8) if masked else None
    w, s = fp8rl.fp8rl_tis_weights_kl(torch.from_numpy(lt).cuda(), torch.from_numpy(lr).cuda(),
                                      None if mask is None else torch.from_numpy(mask).cuda(), clip_c=2.0)
    torch.cuda.synchronize()
    check_tis(w, s, lt, lr, mask, 2.0)


def test_tis_rollout_batch_full_size(fp8rl):
    """32 prompts x 16 samples x 20480 tokens (10.5M, responses of log-uniform length,
    padding masked), C = 2 as in the paper."""
    announce("tis full rollout batch 512 x 20480")
    lt, lr, mask = synth.rollout_logprobs(device="cuda")
    w, s = fp8rl.fp8rl_tis_weights_kl(lt, lr, mask, clip_c=2.0)
    torch.cuda.synchronize()
    _, s_ref = check_tis(w, s, lt.cpu().numpy(), lr.cpu().numpy(), mask.cpu().numpy(), 2.0)
    assert s_ref[3] > 0, "the workload is meant to truncate some weights"


def test_tis_kl_of_two_categoricals(fp8rl):
    """Tokens from the rollout policy p in exact proportions: the GPU's KL estimate
    equals scipy's KL(p || q)."""
    import scipy.stats
    announce("tis categorical KL")
    p = np.array([0.5, 0.25, 0.125, 0.0625, 0.03125, 0.03125])
    q = np.array([0.3, 0.3, 0.2, 0.1, 0.05, 0.05])
    n = 1 << 16
    outcome = np.repeat(np.arange(p.size), (p * n).astype(int))
    lr = np.log(p)[outcome].astype(np.float32)
    lt = np.log(q)[outcome].astype(np.float32)
    _, s = fp8rl.fp8rl_tis_weights_kl(torch.from_numpy(lt).cuda(), torch.from_numpy(lr).cuda())
    s = s.cpu().numpy()
    kl = scipy.stats.entropy(p, q)
    assert abs(s[0] / s[2] - kl) < 1e-6 and abs(s[1] / s[2] - kl) < 1e-6


def test_tis_deterministic_and_other_clip(fp8rl):
    announce("tis determinism, C = 1.5")
    rng = np.random.default_rng(12)
    n = 2_000_003
    lr = torch.from_numpy(-rng.exponential(0.4, n).astype(np.float32)).cuda()
    lt = torch.from_numpy((lr.cpu().numpy() + rng.normal(0, 0.5, n)).astype(np.float32)).cuda()
    w1, s1 = fp8rl.fp8rl_tis_weights_kl(lt, lr, clip_c=1.5)
    w2, s2 = fp8rl.fp8rl_tis_weights_kl(lt, lr, clip_c=1.5)
    torch.cuda.synchronize()
    assert torch.equal(w1, w2) and torch.equal(s1, s2)
    check_tis(w1, s1, lt.cpu().numpy(), lr.cpu().numpy(), None, 1.5)
