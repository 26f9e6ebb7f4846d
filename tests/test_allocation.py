"""Algorithm 1's block-wise delta allocation and the KV I/O model against the
numbers the paper prints (CPU only); see tests/golden/kv_io_table.json."""
import json
import os
from fractions import Fraction

import pytest

from paper_2607_24788_amd import allocation as A

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "kv_io_table.json")


def _golden():
    return json.load(open(GOLDEN))


def test_split_and_assign():
    assert [len(b) for b in A.split(32)] == [11, 10, 11]           # layers 1-11, 12-21, 22-32
    assert sum(A.split(32), []) == list(range(32))
    assert A.candidate_deltas(1024) == [0, 512, 960, 1024]
    d = A.assign(32, 1024, 512)
    assert d[:11] == [0] * 11 and d[11:21] == [512] * 10 and d[21:] == [1024] * 11
    assert A.windows(32, 1024, 512) == [1024] * 11 + [512] * 10 + [0] * 11
    assert A.windows(32, 1024, 0, sizes=(10, 12, 10)) == [1024] * 22 + [0] * 10
    with pytest.raises(ValueError):
        A.split(32, (10, 10, 10))
    with pytest.raises(ValueError):
        A.assign(32, 1024, 2000)


def test_table_kv_io():
    g = _golden()
    m = g["model"]
    L, Hkv, d, e, w = m["n_layers"], m["n_kv_heads"], m["head_dim"], m["elem_bytes"], m["w"]
    deltas = {"0": 0, "w/2": w // 2, "15w/16": 15 * w // 16}
    for row in g["table"]:
        if row["config"] == "vanilla softmax":
            wins = [None] * L
            ctx = row["context"]
        elif row.get("all_linear"):
            wins = [0] * L
            ctx = 32000
        else:
            dm = deltas[row["middle_delta"]]
            # (0, delta, 0) keeps every block's softmax; (0, delta, w) linearises the last block
            wins = A.windows(L, w, dm, sizes=(10, 12, 10))
            if not row.get("last_linear"):
                wins = [w] * 10 + [w - dm] * 12 + [w] * 10
            ctx = 32000
        got = A.kv_io_bytes(wins, ctx, Hkv, d, e) / A.MIB
        assert got == pytest.approx(row["mib"], abs=0.5), row["config"]
    # the 11/10/11 split of the setup section gives 84 / 64 / 46.5 MB
    for dm, want in ((0, 84), (w // 2, 64), (15 * w // 16, 46.5)):
        assert A.kv_io_bytes(A.windows(L, w, dm), 32000, Hkv, d, e) / A.MIB == pytest.approx(want)


def test_reductions_and_motivation_figures():
    g = _golden()
    m = g["model"]
    L, Hkv, d, e, w = m["n_layers"], m["n_kv_heads"], m["head_dim"], m["elem_bytes"], m["w"]
    van = A.kv_io_bytes([None] * L, 32000, Hkv, d, e)
    cfg = {"(0, 0, 0)": [w] * L, "(0, 0, w)": A.windows(L, w, 0, (10, 12, 10)),
           "(0, 15w/16, w)": A.windows(L, w, 15 * w // 16, (10, 12, 10))}
    for name, ratio in g["reductions"].items():
        assert int(van / A.kv_io_bytes(cfg[name], 32000, Hkv, d, e)) == ratio, name
    for row in g["motivation"]:
        wins = [None] * row["softmax_layers"] + [0] * (L - row["softmax_layers"])
        assert A.kv_io_bytes(wins, row["context"], Hkv, d, e) / A.MIB == pytest.approx(row["mib"])


def test_speedup():
    # the ratio form equals the paper's simplified form, exactly
    for alpha in (0, Fraction(1, 2), Fraction(15, 16), 1):
        for w, d in ((1024, 128), (20000, 128), (4096, 4096), (7, 3)):
            assert A.speedup(alpha, w, d) == A.speedup_closed_form(alpha, w, d)
    assert A.speedup(0, 1024, 128) > 1
    # (0, 0, 0) is the reference: alpha = 0 still drops the last block's window
    assert A.speedup(0, 10 ** 12, 1) == pytest.approx(1.5, rel=1e-9)
    # up to 3x in the long-context regime (alpha = 1, w >> d)
    assert A.speedup(1, 10 ** 12, 1) == pytest.approx(_golden()["speedup_max"], rel=1e-9)
    assert A.speedup(1, 10 ** 12, 1) < 3


def test_blockwise_search_picks_the_best_candidate():
    seen = []

    def evaluate(wins):
        seen.append(tuple(wins))
        return -abs(wins[15] - 64)          # prefers the middle window closest to 64

    dm, wins = A.blockwise_search(32, 1024, evaluate)
    assert len(seen) == 4
    assert dm == 960 and wins[11:21] == [64] * 10 and wins[:11] == [1024] * 11 and wins[21:] == [0] * 11


def test_bench_decode_bytes_contain_the_kv_io_model():
    """bench.py's algorithmic decode bytes = the KV I/O model (window K/V of
    every softmax layer) + the per-unit state, token and output terms; the
    state is written once per fold period by default, every step on request."""
    import bench
    from paper_2607_24788_amd import workload as Wm
    for name in ("c2", "c2b", "c3b", "c3", "c5"):
        wl = Wm.workload(name)
        d, Df, G, e = wl.head_dim, wl.feat_dim, wl.G, 2
        units = wl.batch * wl.n_kv_heads
        tok = (2 * d * e + 2 * d * e + 2 * G * d * e + Df * d * 4 + Df * 4) * units * wl.n_layers
        wf = wl.n_layers * d * Df * e
        kv = wl.batch * A.kv_io_bytes(wl.windows, 10 ** 9, wl.n_kv_heads, d, e)
        write = sum((1 if W == 0 else 1 / bench.FOLD_PERIOD) * (Df * d * 4 + Df * 4) * units for W in wl.windows)
        assert bench.decode_bytes(wl, state_write=1) == kv + tok + wf + (Df * d * 4 + Df * 4) * units * wl.n_layers
        assert bench.decode_bytes(wl) == round(kv + tok + wf + write), name


def test_accumulated_kv_io_reproduces_the_figure():
    """Accumulated KV I/O over a 128K-token decode (Sec. IV and its figure of
    KV I/O against sequence length), Llama-3-8B shape, w = 1024, the 10/12/10
    split that reproduces the table's MB/token.  The paper's figures come out
    of this one model under two unit conventions (its "GB" values are 10^12-
    scale):
      caption, (0,0,0):        16.3  = MiB summed over 128,000 tokens / 10^6
      text, (0,15w/16,w):      5.5   = the same convention (the text's 5.5-11.0)
      text, baseline:          "over 17.5" = bytes over 131,072 tokens / 10^12
    The caption's 5.2 for (0,15w/16,w) and the text's 11.0 for (0,0,w) are
    not reproduced (5.48 and 11.22 under the first convention)."""
    sizes = (10, 12, 10)
    acc = lambda wins, n: A.accumulated_kv_io_bytes(wins, n, 8, 128, 2)
    base = [1024] * 32                           # (0, 0, 0): every layer keeps the whole window
    glide = A.windows(32, 1024, 960, sizes)      # (0, 15w/16, w)
    late = A.windows(32, 1024, 0, sizes)         # (0, 0, w): the last block linear
    mib6 = lambda b: b / A.MIB / 1e6
    assert round(mib6(acc(base, 128_000)), 1) == 16.3
    assert round(mib6(acc(glide, 128_000)), 1) == 5.5
    assert 17.5 < acc(base, 131_072) / 1e12 < 17.6
    assert abs(mib6(acc(late, 128_000)) - 11.22) < 0.01
    # closed form against the plain sum of the per-token model, and the warm-up
    for n in (1, 63, 64, 65, 1023, 1024, 1025, 5000):
        assert acc(glide, n) == sum(A.kv_io_bytes(glide, t, 8, 128, 2) for t in range(1, n + 1))
    assert A.accumulated_kv_io_bytes([None], 10, 1, 1, 1) == 2 * sum(range(1, 11))   # full attention: t tokens
