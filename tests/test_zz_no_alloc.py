"""The allocation-free decode attention entry point against the allocating one (GPU).

metro_op_attn_decode_noalloc keeps its descriptors and split states in the
library's fixed device array instead of a per-call allocation.  It must give
bit for bit the output of metro_op_attn_decode on the same inputs, on two
calls in a row (the second smaller, so stale contents of the array from the
first call must not matter), and refuse inputs that need more than the array.
The host block tables are overwritten right after each call returns: the
call must have taken its copy by then.
"""

import numpy as np
import pytest

from oracle import bf16_bits_to_f64
from paper_2411_03519_amd import synth
from tests.test_gpu_attention_ops import build_pool, compare, dev, draw_kv

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def metro():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2411_03519_amd import metro as m
    return m


def case(metro, rng, hd, G, nkv, ctxs):
    nq = G * nkv
    rows = len(ctxs)
    seqs = [draw_kv(rng, int(c), nkv, hd, bool(i % 2)) for i, c in enumerate(ctxs)]
    pool, tables = build_pool(rng, seqs, nkv, hd)
    q = synth.f32_to_bf16_bits(rng.standard_normal((rows, nq, hd)).astype(np.float32) * np.float32(2.0))
    qd, kvd = dev(q), dev(pool)
    bt = np.concatenate(tables).astype(np.int32)
    want = torch.empty(rows * nq * hd, dtype=torch.int16, device="cuda")
    metro.op_attn_decode(qd, kvd, pool.shape[0], nq, nkv, hd, ctxs, bt, want)
    got = torch.full_like(want, -1)
    host_bt = bt.copy()
    host_ctx = np.asarray(ctxs, np.int32).copy()
    metro.lib.metro_op_attn_decode_noalloc(qd.data_ptr(), kvd.data_ptr(), pool.shape[0], nq, nkv, hd, rows,
                                           host_ctx.ctypes.data, host_bt.ctypes.data, got.data_ptr(),
                                           torch.cuda.current_stream().cuda_stream)
    host_bt[:] = rng.permutation(host_bt)          # still valid page ids, in another order
    torch.cuda.synchronize()
    g = got.cpu().numpy().view(np.uint16)
    w = want.cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(g, w)
    # and both against the oracle's attention
    kv = [(bf16_bits_to_f64(k), bf16_bits_to_f64(v), np.array([c - 1])) for (k, v), c in zip(seqs, ctxs)]
    compare(list(g.reshape(rows, 1, nq, hd)), [bf16_bits_to_f64(q)[i][None] for i in range(rows)], kv, G,
            f"no-alloc decode hd {hd} group {G}")


def test_noalloc_decode_matches_allocating_entry_point_twice(metro):
    rng = np.random.default_rng(900)
    # first call: 40 rows of 8 kv heads, contexts up to three 128-page work items
    case(metro, rng, 128, 4, 8, list(rng.integers(1, 4300, 40)))
    # second, smaller call on the same array: other shapes, fewer rows and work items
    case(metro, rng, 64, 2, 2, [1, 17, 300, 2049, 5, 64, 33])


def test_noalloc_decode_rejects_what_exceeds_the_array(metro):
    rows, ctx = 20000, 4096                          # ~670 MB of split states
    q = torch.zeros(64, dtype=torch.int16, device="cuda")
    bt = np.zeros(rows * (ctx // 16), np.int32)
    with pytest.raises(metro.MetroError, match="scratch bytes"):
        metro.op_attn_decode_noalloc(q, q, 1, 32, 8, 128, [ctx] * rows, bt, q)
