"""Layer-wise delta allocation and the per-token KV-cache I/O model.

Host-side configuration tooling for the GLIDE layer (no arithmetic of the
layer itself):

* Algorithm 1 (block-wise delta allocation): SPLIT the stack into early,
  middle and last blocks; ASSIGN delta = 0 to the early block (the whole
  window is softmax) and delta = w to the last (fully linear); the middle
  block takes delta from the candidate set {0, w/2, 15w/16, w}
  (Sec. III-C).  The window the library runs per layer is W_l = w - delta_l
  (the reading of the split index used throughout this repository).  The
  choice among the candidates is made by a caller-supplied evaluation
  (the paper's task-accuracy evaluation is not part of this repository).
* The per-token KV-cache I/O of decode (Sec. II, "Low KV Cache I/O", and the
  KV I/O column of the fine-tuned accuracy table): every softmax layer reads
  its window's keys and values, min(W_l, context) tokens of
  2 * n_kv_heads * head_dim elements; linear-only layers read none.
* The accumulated KV I/O of decoding a sequence token by token (Sec. IV,
  "KV I/O Efficient Reasoning Scalability", and the figure of accumulated KV
  I/O against sequence length): the per-token I/O above summed over the
  tokens, each reading min(W_l, t) tokens while the window fills.
* The theoretical decode speedup of three equal blocks over the (0, 0, 0)
  hybrid baseline (Sec. III-C, "Speedup").
"""
from fractions import Fraction

MIB = 1 << 20


def split(n_layers, sizes=None):
    """SPLIT(M, 3): the three contiguous blocks of a stack of n_layers,
    returned as lists of layer indices.

    ``sizes`` gives the block sizes (early, middle, last).  Default: the
    partition stated in the experimental setup for 32 layers (layers 1-11,
    12-21, 22-32 in 1-indexed terms: 11, 10, 11), generalised as
    (ceil(L/3), L - 2 ceil(L/3), ceil(L/3)) rounded so that the outer blocks
    are equal."""
    if sizes is None:
        e = (n_layers + 2) // 3
        sizes = (e, n_layers - 2 * e, e)
    if len(sizes) != 3 or min(sizes) < 0 or sum(sizes) != n_layers:
        raise ValueError(f"block sizes {sizes} do not partition {n_layers} layers")
    a, b, _ = sizes
    return [list(range(0, a)), list(range(a, a + b)), list(range(a + b, n_layers))]


def candidate_deltas(w):
    """The middle block's search set {0, w/2, 15w/16, w} (Algorithm 1),
    rounded down to whole tokens."""
    return [0, w // 2, (15 * w) // 16, w]


def assign(n_layers, w, middle_delta, sizes=None):
    """ASSIGN: delta_l per layer for the configuration (0, middle_delta, w)."""
    if not 0 <= middle_delta <= w:
        raise ValueError("delta must lie in [0, w]")
    early, middle, last = split(n_layers, sizes)
    delta = [0] * n_layers
    for l in middle:
        delta[l] = middle_delta
    for l in last:
        delta[l] = w
    return delta


def windows(n_layers, w, middle_delta, sizes=None):
    """The per-layer softmax windows W_l = w - delta_l of (0, middle_delta, w)."""
    return [w - d for d in assign(n_layers, w, middle_delta, sizes)]


def blockwise_search(n_layers, w, evaluate, sizes=None):
    """Algorithm 1 with a caller-supplied evaluation: every candidate delta is
    assigned to the middle block, ``evaluate(windows)`` scores the resulting
    configuration, and the best-scoring delta is returned with its windows
    (ties go to the first candidate).  The paper's evaluation is downstream
    task accuracy; any score works here."""
    best = None
    for d in candidate_deltas(w):
        wins = windows(n_layers, w, d, sizes)
        score = evaluate(wins)
        if best is None or score > best[0]:
            best = (score, d, wins)
    return best[1], best[2]


def kv_io_bytes(windows_, context, n_kv_heads, head_dim, elem_bytes=2):
    """KV-cache bytes one decode token reads: each layer reads the keys and
    values of min(W_l, context) tokens (W_l = None: vanilla softmax, the whole
    context)."""
    per_token = 2 * n_kv_heads * head_dim * elem_bytes
    total = 0
    for W in windows_:
        n = context if W is None else min(W, context)
        total += n * per_token
    return total


def accumulated_kv_io_bytes(windows_, n_tokens, n_kv_heads, head_dim, elem_bytes=2):
    """KV-cache bytes read over a whole decode of n_tokens: token t (1-based)
    reads min(W_l, t) cached tokens of every softmax layer (W_l = None: the
    whole context, t tokens).  Per layer that is sum_{t=1..n} min(W, t) =
    n(n+1)/2 for n <= W, else W(W+1)/2 + (n - W) W."""
    per_token = 2 * n_kv_heads * head_dim * elem_bytes
    n = int(n_tokens)
    total = 0
    for W in windows_:
        m = n if W is None else min(W, n)
        total += (m * (m + 1) // 2 + (n - m) * m) * per_token
    return total


def speedup(alpha, w, d):
    """Theoretical decode speedup of (0, alpha w, w) over (0, 0, 0) for three
    equal blocks: the ratio of the per-token costs L w d + L d^2 and
    L w d / 3 + L w (1 - alpha) d / 3 + L d^2.  Exact (Fractions) for
    rational arguments."""
    alpha, w, d = Fraction(alpha), Fraction(w), Fraction(d)
    base = w * d + d * d
    glide = w * d / 3 + w * (1 - alpha) * d / 3 + d * d
    return base / glide


def speedup_closed_form(alpha, w, d):
    """The same speedup in the paper's simplified form
    1 + (1 + alpha) / ((2 + 3 d / w) - alpha)."""
    alpha, w, d = Fraction(alpha), Fraction(w), Fraction(d)
    return 1 + (1 + alpha) / ((2 + 3 * d / w) - alpha)
