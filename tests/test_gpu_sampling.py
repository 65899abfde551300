"""GPU parity of the sampled-verification decision kernels on seeded synthetic
logit rows (war_debug_sample runs them alone), against the oracle's rule on
the very same rows and uniforms.  The kernels decide in fp32 and the oracle in
float64, so a decision may differ only where its margin is below 1e-5
(reported)."""
import numpy as np
import pytest
import torch

from oracle.sampling import filtered_probs, verify_sampled

pytestmark = pytest.mark.gpu


def _case(V, B, k, T, top_k, scale, seed, ties=False):
    from paper_2607_17299_amd import war
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((B * (k + 1), V)) * scale).astype(np.float32)
    if ties:
        # exact ties at the top_k boundary and at the maximum
        for r in range(z.shape[0]):
            order = np.argsort(-z[r].astype(np.float64), kind="stable")
            kth = z[r, order[top_k - 1]]
            z[r, rng.choice(V, 5, replace=False)] = kth
            z[r, rng.choice(V, 2, replace=False)] = z[r].max()
    dls = rng.integers(0, k + 1, B)
    drafts = np.zeros((B, max(k, 1)), np.int32)
    for b in range(B):
        for i in range(dls[b]):
            p = filtered_probs(z[b * (k + 1) + i].astype(np.float64), T, top_k)
            # likely tokens (drawn from the target) and, sometimes, unlikely ones
            drafts[b, i] = rng.choice(V, p=p) if rng.random() < 0.8 else rng.integers(V)
    u = rng.random((B * (k + 1), 2)).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    acc = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    war.debug_sample(dev(z), dev((dls + 1).astype(np.int32)), dev(drafts), k, dev(u), T, top_k, acc, nxt)
    acc, nxt = acc.cpu().numpy(), nxt.cpu().numpy()
    exact, report, n_acc = 0, [], 0
    for b in range(B):
        n = int(dls[b])
        rows = z[b * (k + 1): b * (k + 1) + n + 1].astype(np.float64)
        uu = u[b * (k + 1): b * (k + 1) + n + 1].astype(np.float64)
        r = verify_sampled(rows, drafts[b, :n].tolist(), uu[:, 0], uu[:, 1], T, top_k)
        n_acc += r["accept"]
        if (int(acc[b]), int(nxt[b])) == (r["accept"], r["next"]):
            exact += 1
        else:
            assert min(r["margins"]) < 1e-5, (b, (int(acc[b]), int(nxt[b])), (r["accept"], r["next"]), r["margins"])
            report.append(b)
    return exact, report, n_acc


@pytest.mark.parametrize("V,T,top_k,scale", [
    (151936, 1.0, 200, 1.0),     # the paper's setting on the 36-layer vocabulary
    (151936, 1.0, 200, 6.0),     # peaked rows: drafts are often accepted
    (4096, 0.7, 50, 3.0),
    (4096, 1.5, 4096, 2.0),      # top_k = vocabulary: plain temperature sampling
    (4096, 1.0, 1, 1.0),         # greedy
])
def test_sampling_kernels_match_the_rule(V, T, top_k, scale):
    exact, report, n_acc = _case(V, 24, 4, T, top_k, scale, seed=V + top_k + int(10 * scale))
    assert exact + len(report) == 24 and len(report) <= 1, report
    print(f"\nV={V} T={T} top_k={top_k}: {exact}/24 exact, accepted drafts {n_acc}, reported {report}")


def test_sampling_kernels_ties_at_the_boundary():
    """Exact ties at the top_k boundary (kept by lowest id) and at the maximum."""
    exact, report, _ = _case(4096, 24, 4, 1.0, 200, 2.0, seed=99, ties=True)
    assert exact + len(report) == 24 and len(report) <= 1, report
