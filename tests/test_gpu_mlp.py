"""GPU parity of toc_mlp_epoch (mini-batch gradient descent for the neural network
of section 5.1, first layer on the compressed batch) with the oracle: every step
taken from the GPU's current parameters agrees with the oracle's fp64 step within
1e-5 times each gradient entry's sum of absolute terms; one launch over many batches equals the
same steps launched one by one, bit for bit; argument errors are reported."""

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import config_batches, tiny_batch, Batches

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
U = 2.0 ** -24
NAMES = ("W1", "b1", "W2", "b2", "W3", "b3")


def upload(B):
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    buf = torch.empty(T.toc_upload_size(encs), dtype=torch.uint8, device=DEV)
    return T.toc_upload(encs, buf)


def init(m, h1, h2, C, scale1, seed):
    rng = np.random.default_rng(seed)
    p = {"W1": rng.standard_normal((m, h1)) * scale1, "b1": rng.standard_normal(h1) * 0.1,
         "W2": rng.standard_normal((h1, h2)) * 0.3, "b2": rng.standard_normal(h2) * 0.1,
         "W3": rng.standard_normal((h2, C)) * 0.3, "b3": rng.standard_normal(C) * 0.1}
    return {k: v.astype(np.float32) for k, v in p.items()}


def to_dev(p):
    return {k: torch.from_numpy(v.copy()).to(DEV) for k, v in p.items()}


def to_host(pd):
    return {k: v.cpu().numpy().copy() for k, v in pd.items()}


def check_step(B, b, before, after, labels, lr, worst):
    """after must equal the oracle's step from before, element by element:
    |after - (before - lr g)| <= lr * 1e-5 * S + 4u (|before| + |after|), g the
    oracle's fp64 gradient of the mean loss and S its scale (the sum of the
    absolute values of the terms each gradient entry sums, through the backward
    pass), as 1e-5 * sum |a_ij w_jq| for the products; 4u covers the rounding of
    the update itself."""
    n, rp, c, v = B.batch(b)
    rows = O.canonicalize(n, B.n_cols, rp, c, v)
    r0 = int(B.row_off[b])
    p64 = {k: x.astype(np.float64) for k, x in before.items()}
    want, g = O.mlp_step(rows, B.n_cols, p64, labels[r0:r0 + n], lr)
    S = O.mlp_grad_scale(rows, B.n_cols, p64, labels[r0:r0 + n])
    for k in NAMES:
        a = after[k].astype(np.float64)
        tol = lr * 1e-5 * S[k] + 4 * U * (np.abs(before[k]) + np.abs(a))
        err = np.abs(a - want[k])
        ratio = float(np.max(err / np.maximum(tol, 1e-300), initial=0.0))
        worst[k] = max(worst.get(k, 0.0), ratio)
        assert np.all(err <= tol), f"batch {b} {k}: worst err/tol {ratio:.3g}"


def mixed_set(n_cols):
    parts = []
    for i, spec in enumerate([dict(n_rows=30, density=0.3, n_values=3, prefix_copy=0.7),
                              dict(n_rows=0, density=0.5, n_values=2),
                              dict(n_rows=5, density=0.0, n_values=2),
                              dict(n_rows=120, density=0.2, n_values=2, prefix_copy=0.5),
                              dict(n_rows=1, density=1.0, n_values=1)]):
        rp, c, v = tiny_batch(70 + i, n_cols=n_cols, zeros=(i % 2 == 0), **spec)
        parts.append(Batches(n_cols, [spec["n_rows"]], rp, c, v))
    return Batches.concat(parts)


def deep_set():
    """Dense two-valued rows with copied prefixes: over 16,000 deep codes per batch,
    so the table rows of both first-layer kernels live in the workspace."""
    parts = []
    for k in range(2):
        rp, c, v = tiny_batch(1 + k, n_rows=250, n_cols=400, density=1.0, n_values=2,
                              prefix_copy=0.5)
        parts.append(Batches(400, [250], rp, c, v))
    return Batches.concat(parts)


CASES = {
    # workload batches, h1, h2, classes, first-layer weight scale
    "c3": (lambda: config_batches("c3", 6, 3), 200, 50, 10, 1e-3),
    "c1": (lambda: config_batches("c1", 0, 1), 8, 3, 1, 0.3),
    "c2": (lambda: config_batches("c2", 2, 2), 20, 6, 1, 1.0),
    "c4": (lambda: config_batches("c4", 1, 1), 200, 50, 1, 0.05),
    "mixed_softmax": (lambda: mixed_set(16), 12, 5, 4, 0.3),
    "mixed_sigmoid": (lambda: mixed_set(16), 4, 1, 1, 0.3),
    "deep_rows_in_workspace": (deep_set, 8, 4, 3, 0.05),
    # W2 and W3 too large to stage in LDS beside the tuples: read from global memory
    "wide_hidden": (lambda: config_batches("c5", 3, 2), 400, 60, 3, 0.05),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_each_step_against_oracle(case):
    make, h1, h2, C, s1, = CASES[case]
    B = make()
    dev = upload(B)
    rng = np.random.default_rng(11)
    labels = rng.integers(0, max(C, 2), size=int(B.n_rows.sum())).astype(np.int32)
    ld = torch.from_numpy(labels).to(DEV)
    pd = to_dev(init(B.n_cols, h1, h2, C, s1, 3))
    ws = torch.empty(max(T.toc_mlp_workspace_size(dev, h1, h2, C), 16), dtype=torch.uint8, device=DEV)
    lr, worst = 0.5, {}
    for b in range(B.n_batches):
        before = to_host(pd)
        T.toc_mlp_epoch(dev, pd, ld, lr, ws, b0=b, n_batches=1)
        torch.cuda.synchronize()
        after = to_host(pd)
        if B.n_rows[b] == 0:
            assert all(np.array_equal(after[k], before[k]) for k in NAMES)
        else:
            assert any(not np.array_equal(after[k], before[k]) for k in NAMES)
        check_step(B, b, before, after, labels, lr, worst)
    print(case, {k: f"{v:.3g}" for k, v in worst.items()})


def test_one_launch_equals_steps():
    B = Batches.concat([config_batches("c5", 9, 6), mixed_set(900)])
    dev = upload(B)
    labels = torch.from_numpy(np.random.default_rng(4).integers(0, 3, size=int(B.n_rows.sum()))
                              .astype(np.int32)).to(DEV)
    p0 = init(B.n_cols, 16, 7, 3, 0.2, 8)
    ws = torch.empty(T.toc_mlp_workspace_size(dev, 16, 7, 3), dtype=torch.uint8, device=DEV)
    one = to_dev(p0)
    T.toc_mlp_epoch(dev, one, labels, 0.3, ws)
    steps = to_dev(p0)
    for b in range(B.n_batches):
        T.toc_mlp_epoch(dev, steps, labels, 0.3, ws, b0=b, n_batches=1)
    torch.cuda.synchronize()
    for k in NAMES:
        x, y = one[k].cpu().numpy(), steps[k].cpu().numpy()
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), k
        assert not np.array_equal(x, p0[k]), k


def test_lr_zero_and_errors():
    B = config_batches("c5", 0, 2)
    dev = upload(B)
    labels = torch.zeros(int(B.n_rows.sum()), dtype=torch.int32, device=DEV)
    p0 = init(B.n_cols, 8, 3, 2, 0.2, 1)
    pd = to_dev(p0)
    ws = torch.empty(T.toc_mlp_workspace_size(dev, 8, 3, 2), dtype=torch.uint8, device=DEV)
    T.toc_mlp_epoch(dev, pd, labels, 0.0, ws)
    torch.cuda.synchronize()
    assert all(np.array_equal(pd[k].cpu().numpy(), p0[k]) for k in NAMES)
    for kw in (dict(b0=1, n_batches=2), dict(b0=-1, n_batches=1)):
        with pytest.raises(T.TocError) as ei:
            T.toc_mlp_epoch(dev, pd, labels, 0.1, ws, **kw)
        assert ei.value.status == T.TOC_EINVAL
    for lr in (float("nan"), float("inf")):
        with pytest.raises(T.TocError) as ei:
            T.toc_mlp_epoch(dev, pd, labels, lr, ws)
        assert ei.value.status == T.TOC_EINVAL
    with pytest.raises(T.TocError) as ei:           # h1 not a multiple of 4
        T.toc_mlp_epoch(dev, to_dev(init(B.n_cols, 6, 3, 2, 0.2, 1)), labels, 0.1, ws)
    assert ei.value.status == T.TOC_EUNSUPPORTED
    with pytest.raises(T.TocError) as ei:           # workspace too small
        T.toc_mlp_epoch(dev, pd, labels, 0.1, ws[:16])
    assert ei.value.status == T.TOC_ESIZE
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    hbuf = np.zeros(T.toc_upload_size(encs, T.TOC_UPLOAD_HOST), np.uint8)
    hdev = T.toc_upload(encs, hbuf, T.TOC_UPLOAD_HOST)
    with pytest.raises(T.TocError) as ei:
        T.toc_mlp_epoch(hdev, pd, labels, 0.1, ws)
    assert ei.value.status == T.TOC_EINVAL
