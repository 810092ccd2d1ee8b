"""The allocation-free decode step (fp_decode_step_noalloc) against fp_decode_step: same
outputs bit for bit, on consecutive calls that share the library's static scratch
region, the later ones with a smaller batch (and a single sequence, which takes the
single-sequence schedule)."""
import pytest

from fpgen.workloads import Shape
from tests.gpu_harness import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2501_13111_amd as P
    P.load()
    yield


def _run(shape, wq, kvq, B, P, steps, noalloc, seed=12):
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal
    H = shape.hidden
    with Fingerprint(shape, wq, kvq, seed=seed) as fp:
        fp.set_decode_graph(False)
        x = torch.empty(B * P * H, dtype=torch.bfloat16, device="cuda")
        fill_normal(x, seed, -1, 15, 0.0, 1.0)
        y = torch.empty_like(x)
        fp.prefill(x, y, B, P)
        a = y.view(B, P, H)[:, -1, :].contiguous()
        b = torch.empty_like(a)
        outs = []
        for _ in range(steps):
            (fp.decode_step_noalloc if noalloc else fp.decode_step)(a, b)
            outs.append(b.clone())
            a, b = b, a
        torch.cuda.synchronize()
        return torch.stack(outs).cpu()


CASES = [
    ("int4-int8kv-gqa", Shape(2, 512, 8, 2, 64, 768, 6, 40, 48), "int4", "int8"),
    ("bf16", Shape(2, 512, 4, 4, 128, 640, 6, 40, 48), "bf16", "bf16"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_noalloc_decode_matches_decode_step(case):
    import torch
    name, shape, wq, kvq = case
    for B in (6, 3, 1):               # consecutive calls, each with a smaller input
        log(f"noalloc {name} B={B}")
        want = _run(shape, wq, kvq, B, 40, 4, noalloc=False)
        got = _run(shape, wq, kvq, B, 40, 4, noalloc=True)
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), (name, B)


def test_noalloc_decode_at_full_size_batch():
    """The 70B shard's decode schedule (64 sequences, int4 weights, int8 cache, GQA 8:1) at a
    short prompt: the largest scratch of the workloads."""
    import torch
    shape = Shape(1, 8192, 8, 1, 128, 3584, 64, 16, 20)
    for B in (64, 17):
        log(f"noalloc 70b-shard-layer B={B}")
        want = _run(shape, "int4", "int8", B, 16, 2, noalloc=False)
        got = _run(shape, "int4", "int8", B, 16, 2, noalloc=True)
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), B
