"""The attention kernels on their own against the oracle's attention (GPU).

metro_op_attn_decode / metro_op_attn_prefill run the model's decode and
chunked-prefill attention kernels (same launchers, same work split) on caller
buffers: bf16 q and a pool of KV pages written here in the layout metro_ops.h
states, with each sequence's pages scattered over the pool.  The reference is
``oracle.causal_gqa_attention`` on the same bf16 values in float64, rounded to
bf16 at the output as the precision contract does.

Bound per element: one bf16 ulp of the reference (the GPU's fp32 result and
the exact value may round to neighbouring bf16 values) plus the error of the
softmax weights in the matrix cores, which take p as the pair hi = bf16(p),
lo = bf16(p - hi): |p - hi - lo| <= 2^-16 p, so the weighted mean of v moves by
at most 2^-16 max|v| -- taken here as 2^-14 max|v| to cover the fp32 score,
exp2 and accumulation roundings as well.  The fraction of elements equal to
the reference bit for bit is reported and must stay above 97%.

Cases: every head dim / group pair the model accepts (64 and 128 x 1, 2, 4,
8), contexts on both sides of a page (16 keys), of a 128-page work item (2048
keys, the decode split) and of the 512 page ids the prefill kernel stages in
LDS (8192 keys); softmax inputs from flat to sharply peaked, and keys whose
scores rise along the context so the running maximum moves page after page.
Every slot of the pool that holds no key of a sequence is filled with NaN and
Inf bit patterns, so a masked key that leaked into a sum would show.
"""

import numpy as np
import pytest

from oracle import bf16_bits_to_f64, bf16_round, causal_gqa_attention
from paper_2411_03519_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

PAIRS = [(hd, g) for hd in (64, 128) for g in (1, 2, 4, 8)]


@pytest.fixture(scope="module")
def metro():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2411_03519_amd import metro as m
    return m


def say(*a):
    print(*a, flush=True)


def tile_offsets(hd):
    """Element offsets of (key r, dim e) inside a K tile and a V^T tile (metro_ops.h)."""
    r, e = np.meshgrid(np.arange(16), np.arange(hd), indexing="ij")
    k = ((e // 32 * 4 + (e // 8) % 4) * 16 + r) * 8 + e % 8
    v = ((e // 32 * 4 + r // 4) * 16 + e % 16) * 8 + ((e // 16) % 2) * 4 + r % 4
    return k, v


def draw_kv(rng, ctx, nkv, hd, rising=False):
    """bf16 bits of K, V [ctx, nkv, hd]; with rising, later keys have larger norms."""
    k = rng.standard_normal((ctx, nkv, hd)).astype(np.float32)
    if rising:
        k *= (1.0 + 3.0 * np.arange(ctx, dtype=np.float32) / max(ctx, 1))[:, None, None]
    v = rng.standard_normal((ctx, nkv, hd)).astype(np.float32)
    return synth.f32_to_bf16_bits(k), synth.f32_to_bf16_bits(v)


def build_pool(rng, seqs_kv, nkv, hd, spare=7):
    """Scatter the sequences' pages over a pool; returns (pool bits [n_pages, 2, nkv, 16*hd],
    block tables per sequence).  Slots no sequence owns hold NaN and Inf bit
    patterns (what a fresh or reused page may hold): masked keys must
    contribute exactly nothing."""
    need = [(len(k) + 15) // 16 for k, _ in seqs_kv]
    n_pages = sum(need) + spare
    ids = rng.permutation(n_pages)
    pool = rng.choice(np.array([0x7FC0, 0xFFC1, 0x7F80, 0xFF80], np.uint16), size=(n_pages, 2, nkv, 16 * hd))
    koff, voff = tile_offsets(hd)
    tables, at = [], 0
    for (k, v), npg in zip(seqs_kv, need):
        tab = ids[at:at + npg]
        at += npg
        tables.append(tab)
        for j, pid in enumerate(tab):
            kk, vv = k[16 * j:16 * j + 16], v[16 * j:16 * j + 16]
            n = len(kk)
            for h in range(nkv):
                pool[pid, 0, h, koff[:n].ravel()] = kk[:, h, :].ravel()
                pool[pid, 1, h, voff[:n].ravel()] = vv[:, h, :].ravel()
    return pool, tables


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


def compare(got_bits, q_rows, kv_of_row, group, what):
    """Sequence by sequence: got_bits[i] [n, nq, hd] bf16 bits of the GPU's
    output for queries q_rows[i] [n, nq, hd] at positions qpos over keys
    kv_of_row[i] = (K, V, qpos) (float64 values of the bf16 inputs)."""
    n_exact = n_all = 0
    worst = 0.0
    for i, (qi, (K, V, qpos)) in enumerate(zip(q_rows, kv_of_row)):
        ref = causal_gqa_attention(qi, K, V, qpos)                  # float64 [n, nq, hd]
        want = bf16_round(ref)
        g = bf16_bits_to_f64(got_bits[i])
        vmax = np.abs(V).max(axis=(0, 2))                            # per kv head
        vm = np.repeat(vmax, group)[None, :, None]
        _, e = np.frexp(np.maximum(np.abs(ref), 2.0 ** -126))
        ulp = np.ldexp(1.0, e - 8)
        bound = ulp + vm * 2.0 ** -14
        err = np.abs(g - want)
        assert np.all(err <= bound), f"{what}: row {i} error {err.max():.3e} over bound at {np.argmax(err - bound)}"
        worst = max(worst, float(np.max(err / bound)))
        n_exact += int(np.sum(g == want))
        n_all += g.size
    frac = n_exact / n_all
    say(f"{what}: {n_all} outputs, {100 * frac:.2f}% bit-exact, worst error {worst:.3f} of the bound")
    assert frac >= 0.97, f"{what}: only {100 * frac:.2f}% bit-exact"


def run_decode(metro, rng, hd, G, nkv, ctxs, scales, rising):
    nq = G * nkv
    rows = len(ctxs)
    seqs = [draw_kv(rng, c, nkv, hd, r) for c, r in zip(ctxs, rising)]
    pool, tables = build_pool(rng, seqs, nkv, hd)
    q = np.stack([synth.f32_to_bf16_bits(rng.standard_normal((nq, hd)).astype(np.float32) * np.float32(s))
                  for s in scales])
    out = torch.empty(rows * nq * hd, dtype=torch.int16, device="cuda")
    metro.op_attn_decode(dev(q), dev(pool), pool.shape[0], nq, nkv, hd, ctxs, np.concatenate(tables), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16).reshape(rows, 1, nq, hd)
    q64 = bf16_bits_to_f64(q)
    kv = [(bf16_bits_to_f64(k), bf16_bits_to_f64(v), np.array([c - 1])) for (k, v), c in zip(seqs, ctxs)]
    return got, [q64[i][None] for i in range(rows)], kv


@pytest.mark.parametrize("hd,G", PAIRS)
def test_decode_attention_every_head_dim_and_group(metro, hd, G):
    rng = np.random.default_rng(100 + hd + G)
    nkv = 2
    ctxs = [1, 15, 16, 17, 33, 250, 2047, 2049]
    scales = [0.3, 1.0, 2.0, 4.0, 0.5, 3.0, 1.0, 6.0]
    rising = [False, True, False, True, False, True, True, False]
    got, q, kv = run_decode(metro, rng, hd, G, nkv, ctxs, scales, rising)
    compare(list(got), q, kv, G, f"decode hd {hd} group {G}")


@pytest.mark.parametrize("G", [4, 8])
def test_decode_attention_llama_shapes_long_contexts(metro, G):
    # 8 kv heads of dim 128 (Llama-3 8B: group 4, 70B: group 8), contexts across
    # one, two and three 128-page work items, scattered pages
    rng = np.random.default_rng(200 + G)
    ctxs = [1, 2048, 2049, 4096, 4300, 1300, 16, 4097]
    scales = [1.0, 2.0, 1.0, 4.0, 0.7, 8.0, 1.5, 3.0]
    rising = [False, True, False, True, True, False, False, True]
    got, q, kv = run_decode(metro, rng, 128, G, 8, ctxs, scales, rising)
    compare(list(got), q, kv, G, f"decode 8 kv heads group {G}")


def test_decode_attention_many_rows(metro):
    # more than 512 workgroups: the kernel variant with one page in flight per wave
    rng = np.random.default_rng(300)
    ctxs = list(rng.integers(1, 400, 80))
    assert sum((c + 15) // 16 for c in ctxs) > 0 and len(ctxs) * 8 > 512
    scales = list(rng.uniform(0.3, 5.0, 80))
    rising = list(rng.integers(0, 2, 80).astype(bool))
    got, q, kv = run_decode(metro, rng, 128, 4, 8, ctxs, scales, rising)
    compare(list(got), q, kv, 4, "decode 80 rows x 8 kv heads")


def run_prefill(metro, rng, hd, G, nkv, items, scale=1.5):
    """items: (keys before the chunk, chunk queries, rising keys)."""
    nq = G * nkv
    seqs = [draw_kv(rng, b + c, nkv, hd, r) for b, c, r in items]
    pool, tables = build_pool(rng, seqs, nkv, hd)
    cu = np.concatenate([[0], np.cumsum([c for _, c, _ in items])]).astype(np.int32)
    T = int(cu[-1])
    q = synth.f32_to_bf16_bits(rng.standard_normal((T, nq, hd)).astype(np.float32) * np.float32(scale))
    out = torch.empty(T * nq * hd, dtype=torch.int16, device="cuda")
    metro.op_attn_prefill(dev(q), dev(pool), pool.shape[0], nq, nkv, hd, cu, [b for b, _, _ in items],
                          np.concatenate(tables), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16).reshape(T, nq, hd)
    q64 = bf16_bits_to_f64(q)
    rows, kv = [], []
    for i, ((b, c, _), (k, v)) in enumerate(zip(items, seqs)):
        rows.append(q64[cu[i]:cu[i + 1]])
        kv.append((bf16_bits_to_f64(k), bf16_bits_to_f64(v), np.arange(b, b + c)))
    gots = [got[cu[i]:cu[i + 1]] for i in range(len(items))]
    return gots, rows, kv


@pytest.mark.parametrize("hd,G", PAIRS)
def test_prefill_attention_every_head_dim_and_group(metro, hd, G):
    rng = np.random.default_rng(400 + hd + G)
    items = [(0, 1, False), (0, 23, True), (19, 40, False), (300, 64, True), (0, 300, False), (16, 16, True)]
    gots, rows, kv = run_prefill(metro, rng, hd, G, 2, items)
    compare(gots, rows, kv, G, f"prefill hd {hd} group {G}")


@pytest.mark.parametrize("G", [4, 8])
def test_prefill_attention_llama_shapes(metro, G):
    # 8 kv heads of dim 128; a 512-token chunk after 1000 keys, a chunk whose
    # context passes the 512 page ids staged in LDS, ragged short chunks
    rng = np.random.default_rng(500 + G)
    items = [(1000, 512, True), (8300, 64, False), (0, 17, False), (2040, 9, True), (511, 1, False)]
    gots, rows, kv = run_prefill(metro, rng, 128, G, 8, items, scale=2.0)
    compare(gots, rows, kv, G, f"prefill 8 kv heads group {G}")


def test_attention_ops_reject_bad_arguments(metro):
    q = torch.zeros(64 * 128, dtype=torch.int16, device="cuda")
    kv = torch.zeros(4 * 2 * 8 * 16 * 128, dtype=torch.int16, device="cuda")
    out = torch.zeros_like(q)
    with pytest.raises(metro.MetroError, match="page id"):
        metro.op_attn_decode(q, kv, 4, 32, 8, 128, [20], [0, 4], out)
    with pytest.raises(metro.MetroError, match="group"):
        metro.op_attn_decode(q, kv, 4, 24, 8, 128, [20], [0, 1], out)
    with pytest.raises(metro.MetroError, match="queries"):
        metro.op_attn_prefill(q, kv, 4, 32, 8, 128, [0, 0], [3], [0], out)
