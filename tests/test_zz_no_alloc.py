"""The layer forward that allocates nothing (seer_layer_forward_varlen_noalloc,
whose workspace is a device array inside the library) against
seer_layer_forward_varlen with a caller workspace: same kernels, same inputs,
so outputs and counts must be identical bit for bit.  Two calls in a row, the
second with fewer rows (the shared array keeps the first call's contents),
then a rows bound beyond the array is refused."""
import numpy as np
import pytest

from gpu_util import dev, host, log, upload_weights

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    from paper_2607_14557_amd import seer
    seer.load_library()
    return seer


def _layer(S, d, H, dh, I, dtype, rng):
    import torch
    from paper_2607_14557_amd.runner import dims_for
    from workloads.generate import round_to_dtype
    W = {k: round_to_dtype(rng.standard_normal(shape) * 0.02, dtype) for k, shape in
         (("wq", (d, d)), ("wk", (d, d)), ("wv", (d, d)), ("wo", (d, d)), ("wg", (I, d)), ("wu", (I, d)),
          ("wd", (d, I)))}
    W.update(g1=np.ones(d), g2=np.ones(d))
    dims = dims_for(d, H, dh, I, dtype)
    packed = torch.empty(S.seer_prepacked_bytes(dims), dtype=torch.uint8, device="cuda")
    S.seer_prepack_weights(dims, upload_weights(W, dtype), packed)
    return dims, packed


def _compare(S, dims, packed, dtype, lens, rows_ub, rng, eps):
    import torch
    d = dims.d_model
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    T = int(cu[-1])
    x = np.zeros((rows_ub, d))
    x[:T] = rng.standard_normal((T, d))
    xd, cud = dev(x, dtype), dev(cu)
    used = dev(np.maximum(np.asarray(lens) - 1, 0))          # a padded tail per sequence (seqused)
    ws = torch.empty(S.seer_layer_workspace_bytes(dims, rows_ub), dtype=torch.uint8, device="cuda")
    y_ref = torch.zeros_like(xd)
    c_ref = torch.zeros(rows_ub, dtype=torch.int32, device="cuda")
    S.seer_layer_forward_varlen(dims, packed, xd, y_ref, rows_ub, cud, used, len(lens), eps, c_ref, ws)
    y = torch.full_like(xd, 7.0)
    c = torch.full((rows_ub,), -5, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    S.seer_layer_forward_varlen_noalloc(dims, packed, xd, y, rows_ub, cud, used, len(lens), eps, c, status)
    torch.cuda.synchronize()
    assert torch.equal(y[:T], y_ref[:T]), "outputs differ"
    assert torch.equal(c[:T], c_ref[:T]), "counts differ"
    assert torch.all(y[T:] == 7.0), "rows past cu[B] must not be written"
    assert int(status.item()) == 0
    log("  %s lens %s: outputs and counts identical (rows bound %d)" % (dtype, list(lens), rows_ub))
    return host(c_ref[:T])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_point(S, dtype):
    rng = np.random.default_rng(21)
    d, H, dh, I = (512, 4, 128, 1024) if dtype == "bf16" else (256, 4, 64, 688)
    dims, packed = _layer(S, d, H, dh, I, dtype, rng)
    eps = 0.01 * 0.0004 * d
    c1 = _compare(S, dims, packed, dtype, [300, 77, 513, 1, 129], 1100, rng, eps)
    c2 = _compare(S, dims, packed, dtype, [40, 3, 90], 140, rng, eps)
    assert c1.sum() > 0 and c2.sum() > 0


def test_noalloc_llada_shape_and_limit(S):
    """The LLaDA-8B layer shape at the row count of a cached truncated step
    (B=16, 1592 kept window rows), then a smaller call, then a rows bound
    whose workspace exceeds the 256 MiB array (refused, nothing launched)."""
    import torch
    from paper_2607_14557_amd.runner import dims_for
    rng = np.random.default_rng(22)
    d, H, dh, I = 4096, 32, 128, 12288
    dims = dims_for(d, H, dh, I, "bf16")
    g = torch.Generator(device="cuda").manual_seed(3)
    Wd = {k: (torch.randn(shape, generator=g, device="cuda") * 0.02).to(torch.bfloat16) for k, shape in
          (("wq", (d, d)), ("wk", (d, d)), ("wv", (d, d)), ("wo", (d, d)), ("wg", (I, d)), ("wu", (I, d)),
           ("wd", (d, I)))}
    Wd.update(g1=torch.ones(d, device="cuda"), g2=torch.ones(d, device="cuda"))
    packed = torch.empty(S.seer_prepacked_bytes(dims), dtype=torch.uint8, device="cuda")
    S.seer_prepack_weights(dims, Wd, packed)
    del Wd
    eps = 0.01 * 0.0004 * d
    lens = rng.integers(17, 90, size=16)
    lens[0] += 1592 - int(lens.sum())
    _compare(S, dims, packed, "bf16", lens, 1792, rng, eps)
    _compare(S, dims, packed, "bf16", [300, 100], 512, rng, eps)
    assert S.seer_layer_workspace_bytes(dims, 2730) <= (256 << 20) < S.seer_layer_workspace_bytes(dims, 2731)
    x = torch.zeros(2731, d, dtype=torch.bfloat16, device="cuda")
    cu = dev(np.array([0, 2731]))
    with pytest.raises(S.SeerError) as ei:
        S.seer_layer_forward_varlen_noalloc(dims, packed, x, torch.empty_like(x), 2731, cu, None, 1, 0.0, None)
    assert ei.value.code == S.SEER_EWORKSPACE
