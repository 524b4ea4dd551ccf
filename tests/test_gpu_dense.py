"""GPU parity of full_attention (the dense baseline: softmax of the Eq. 4 scores over
every row, then the weighted value sum) against the oracle's float64 attention over
all rows, for dtypes, head dims, GQA groups, lengths that are not multiples of the
kernel's chunk, a single row, and two sequences."""
import math
import zlib

import numpy as np
import pytest

from gpu_harness import OUT_TOL, handle_of, rel_err, to_dev, torch_cuda
from oracle import oracle as O
from paper_2607_27692_amd import retopk as R
from paper_2607_27692_amd.inputs import bf16_bits_to_f32, to_bf16_bits

pytestmark = pytest.mark.gpu

CASES = [
    # dtype, d, B, Hq, Hkv, L
    ("f32", 64, 1, 1, 1, 2049),
    ("f32", 128, 1, 4, 2, 3001),
    ("bf16", 128, 1, 32, 8, 16385),
    ("bf16", 128, 2, 8, 1, 9000),
    ("bf16", 64, 1, 4, 4, 5000),
    ("bf16", 128, 1, 4, 1, 1),
    ("bf16", 128, 1, 8, 4, 1024),
    # group sizes that are not powers of two (padded groups)
    ("bf16", 128, 1, 28, 4, 9000),
    ("bf16", 64, 2, 6, 2, 4097),
    ("f32", 128, 1, 10, 2, 3000),
    # the 8-head build at d = 64, bf16 and fp32
    ("bf16", 64, 1, 8, 1, 3000),
    ("f32", 64, 1, 16, 2, 2500),
]


@pytest.mark.parametrize("dtype,d,B,Hq,Hkv,L", CASES)
def test_full_attention_parity(dtype, d, B, Hq, Hkv, L):
    torch = torch_cuda()
    print(f"full attention {dtype} d={d} B={B} Hq={Hq} Hkv={Hkv} L={L}", flush=True)
    rng = np.random.default_rng(zlib.crc32(f"{dtype}-{d}-{B}-{Hq}-{Hkv}-{L}".encode()))
    q = rng.standard_normal((B, Hq, d)).astype(np.float32) * math.sqrt(d) / 2
    k = rng.standard_normal((B, Hkv, L, d)).astype(np.float32)
    v = rng.standard_normal((B, Hkv, L, d)).astype(np.float32)
    if dtype == "bf16":
        raw = [to_bf16_bits(x) for x in (q, k, v)]
        q, k, v = [bf16_bits_to_f32(x) for x in raw]
    else:
        raw = [q, k, v]
    p = O.Params(B, Hq, Hkv, d, L, 16, 0, 1, 0, 0.5, 0)
    h = handle_of(p, dtype)
    qd, kd, vd = (to_dev(x) for x in raw)
    out = torch.full((B, Hq, d), float("nan"), dtype=torch.float32, device="cuda")
    h.full(qd, kd, vd, L, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    h.close()
    G = Hq // Hkv
    worst = 0.0
    for b in range(B):
        for hq in range(Hq):
            ref = O.attend(q[b, hq], k[b, hq // G], v[b, hq // G], np.arange(L))
            e = rel_err(got[b, hq], ref)
            worst = max(worst, e)
            assert e <= OUT_TOL[dtype], f"b={b} h={hq}: relative error {e:.3g}"
    print(f"max relative error {worst:.3g}", flush=True)


def test_stream_read_runs():
    """The streaming-read measurement aid reads a buffer and leaves the sink alone
    (the fold of a buffer of equal words is 0, not the sentinel)."""
    torch = torch_cuda()
    x = torch.ones(1 << 20, dtype=torch.float32, device="cuda")
    sink = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    R.retopk_stream_read(x, x.numel() * 4, sink)
    torch.cuda.synchronize()
    assert int(sink.item()) == 7
