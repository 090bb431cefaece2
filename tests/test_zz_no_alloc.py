"""The allocation-free fit solve (scd_fit_solve_noalloc) against the workspace solve
(scd_fit_solve) through the C ABI.

The two share the solve kernel; the allocation-free call keeps the fp64 matrices in the library's
device-resident scratch array and splits the layers over as many launches as that array needs.
The per-layer arithmetic is the same, so the outputs must be bit-identical.  Two calls in a row:
the first with enough w = 256 layers to need two launches, the second with a smaller model, so a
stale scratch array from the first call would show.
"""
import pytest
import torch

import paper_2606_07684_amd as scd

pytestmark = pytest.mark.gpu


def _model(L, heads, head_dim, rank):
    return scd.Model(n_layers=L, d_model=256, n_kv_heads=heads, head_dim=head_dim,
                     rope_theta=1e4, dtype="bf16", is_patch=[0] * L, rank_k=[rank] * L,
                     rank_v=[rank] * L, rank_h=[32] * L)


def _sums(model, n_rows, seed, dev):
    """Gram and column sums of seeded rows with a decaying spectrum (host fp64, rounded once)."""
    w2 = 2 * model.basis_width
    gen = torch.Generator().manual_seed(seed)
    scale = 1.0 / torch.arange(1, w2 + 1, dtype=torch.float64)
    gram, colsum = [], []
    for _ in range(model.n_layers):
        x = torch.randn(n_rows, w2, generator=gen, dtype=torch.float64) * scale + 0.1
        gram.append((x.T @ x).float().to(dev))
        colsum.append(x.sum(0).float().to(dev))
    return gram, colsum


def _outputs(model, dev):
    L, w, r = model.n_layers, model.basis_width, model.rank_k[0]
    nan = float("nan")
    mk = lambda *shape: [torch.full(shape, nan, dtype=torch.bfloat16, device=dev)
                         for _ in range(L)]
    return mk(r, w), mk(w, r), mk(w), mk(w)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    scd.load_library()
    yield
    torch.cuda.synchronize()


def test_noalloc_solve_matches_workspace_solve_twice():
    dev = torch.device("cuda")
    assert scd.scd_fit_solve_noalloc_max_bytes() == 64 << 20
    # (layers, heads, head_dim, rank, rows): 11 layers at w = 256 need 8.4 MB each, so the
    # scratch array takes 7 per launch and the call makes two launches; the second call is smaller.
    cases = [(11, 2, 128, 64, 2000), (3, 2, 64, 32, 700)]
    for i, (L, heads, hd, rank, n_rows) in enumerate(cases):
        model = _model(L, heads, hd, rank)
        gram, colsum = _sums(model, n_rows, 100 + i, dev)
        lam = 0.05 * n_rows
        for branch in (scd.FIT_KEYS, scd.FIT_VALUES):
            print(f"[noalloc] call {i}: L={L} w={model.basis_width} rank={rank} "
                  f"branch={branch}", flush=True)
            ref = _outputs(model, dev)
            ws = torch.empty(scd.scd_fit_workspace_bytes(model, n_rows), dtype=torch.uint8,
                             device=dev)
            scd.scd_fit_solve(model, branch, n_rows, lam, True, gram, colsum, *ref, ws)
            got = _outputs(model, dev)
            scd.scd_fit_solve_noalloc(model, branch, n_rows, lam, True, gram, colsum, *got)
            torch.cuda.synchronize()
            for name, a, b in zip(("w_enc", "w_dec", "mu_enc", "mu_dec"), ref, got):
                for l in range(L):
                    assert torch.isfinite(a[l].float()).all(), f"{name}[{l}] not finite"
                    assert torch.equal(a[l], b[l]), f"call {i} {name}[{l}] differs"
