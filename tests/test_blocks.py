"""The combinator front end (blocks.py, Section 3 of the paper).

CPU: the op table each expression enumerates; the graphs traced for the paper's three shapes (the recursive
Tree-LSTM over binary trees with a forward declaration, a text pipeline folding an LSTM over words, a balanced
Reduce of embedded tokens) evaluated by the oracle against a direct recursion over the same Python inputs with
the oracle's per-node cells (independent of the compiler's graph); Reduce's split at floor(n / 2); Optional.
GPU: a compiled batch of random trees through the C ABI against the oracle, forward and backward.
"""
import numpy as np
import pytest

from oracle import cells as OC
from oracle import evaluate as EV
from paper_1702_02181_amd import blocks as B
from paper_1702_02181_amd import gen
from tests._helpers import oracle_batch, oracle_params

TL, LS, RNN, EMB = gen.KIND_TREELSTM, gen.KIND_LSTM, gen.KIND_TREERNN, gen.KIND_EMBED


def tree_lstm_expr():
    """The recursive sentiment model: a leaf is TreeLSTM(word row, 0, 0), a pair TreeLSTM(0, left, right)."""
    expr = B.ForwardDeclaration()
    word = B.AllOf(B.Scalar(), B.Zeros())
    pair = B.AllOf(B.Zeros(), B.Record([(0, expr()), (1, expr())]))
    expr_def = B.OneOf(key_fn=lambda t: isinstance(t, tuple), cases={False: word, True: pair}) >> B.Op(TL, 0)
    expr.resolve_to(expr_def)
    return expr()


def random_tree(rng, n_leaves, vocab):
    if n_leaves == 1:
        return int(rng.integers(0, vocab))
    k = int(rng.integers(1, n_leaves))
    return (random_tree(rng, k, vocab), random_tree(rng, n_leaves - k, vocab))


def _params(H, specs, dtype="f32", seed=0):
    rng = np.random.default_rng(seed)
    return [gen.make_param_set(rng, kind, in_dim, arity, H, dtype) for kind, in_dim, arity in specs]


def _oracle_states(w):
    f = EV.forward(oracle_batch(w), oracle_params(w), w.hidden, w.leaf_table)
    return f["h"]


def _direct_tree_lstm(t, P, H, table):
    """h, c of a nested-tuple tree by recursion with the oracle's cell (no graph, no schedule)."""
    if not isinstance(t, tuple):
        h, c, _ = OC.forward_node(TL, P, H, table[t].astype(np.float64), [np.zeros(H), np.zeros(H)],
                                  [np.zeros(H), np.zeros(H)])
        return h, c
    (hl, cl), (hr, cr) = _direct_tree_lstm(t[0], P, H, table), _direct_tree_lstm(t[1], P, H, table)
    h, c, _ = OC.forward_node(TL, P, H, None, [hl, hr], [cl, cr])
    return h, c


def test_op_table_of_the_tree_lstm_expression():
    c = B.Compiler(tree_lstm_expr())
    assert c.ops == [gen.OpSpec(TL, 0, 1, 0), gen.OpSpec(TL, 2, 0, 0)]


def test_recursive_tree_lstm_matches_direct_recursion():
    rng = np.random.default_rng(1)
    H, V = 6, 30
    trees = [random_tree(rng, int(n), V) for n in (1, 2, 5, 9, 17)]
    table = 0.5 * rng.standard_normal((V, H)).astype(np.float32)
    params = _params(H, [(TL, H, 2)])
    w, outs = B.Compiler(tree_lstm_expr()).build(trees, params, H, table)
    h = _oracle_states(w)
    P = oracle_params(w)[0]
    for t, out in zip(trees, outs):
        want, _ = _direct_tree_lstm(t, P, H, table)
        np.testing.assert_allclose(h[out.id], want, rtol=1e-12, atol=1e-14)
    # every graph has exactly one root, its output
    assert gen.count_roots(w.num_nodes, w.child_idx) == len(trees)


def test_text_pipeline_folds_an_lstm_over_words():
    vocab = {w: i for i, w in enumerate("the cat sat on a mat and dog ran".split())}
    H = 5
    text2vec = (B.InputTransform(str.split) >> B.Map(B.InputTransform(vocab.get) >> B.Scalar()) >>
                B.Fold(B.Op(LS, 0)))
    c = B.Compiler(text2vec)
    assert c.ops == [gen.OpSpec(LS, 1, 1, 0)]
    sents = ["the cat sat on a mat", "dog ran", "a"]
    rng = np.random.default_rng(2)
    table = rng.standard_normal((len(vocab), H)).astype(np.float32)
    params = _params(H, [(LS, H, 1)])
    w, outs = c.build(sents, params, H, table)
    # a chain per sentence: node i reads word i and its predecessor (the first one the zero state)
    gp = w.graph_ptr
    for g, s in enumerate(sents):
        words = s.split()
        nodes = range(gp[g], gp[g + 1])
        assert [int(w.node_input[v]) for v in nodes] == [vocab[x] for x in words]
        assert [int(w.child_idx[w.child_ptr[v]]) for v in nodes] == [-1] + list(nodes)[:-1]
        assert outs[g].id == gp[g + 1] - 1
    h = _oracle_states(w)
    P = oracle_params(w)[0]
    for g, s in enumerate(sents):
        hs, cs = np.zeros(H), np.zeros(H)
        for x in s.split():
            hs, cs, _ = OC.forward_node(LS, P, H, table[vocab[x]].astype(np.float64), [hs], [cs])
        np.testing.assert_allclose(h[outs[g].id], hs, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 8])
def test_reduce_is_balanced_at_floor_half(n):
    H = 4
    red = B.Map(B.Scalar() >> B.Op(EMB, 0)) >> B.Reduce(B.Op(RNN, 1))
    c = B.Compiler(red)
    assert c.ops == [gen.OpSpec(EMB, 0, 1, 0), gen.OpSpec(RNN, 2, 0, 1)]
    rng = np.random.default_rng(n)
    table = rng.standard_normal((10, H)).astype(np.float32)
    params = [gen.ParamSet(EMB, H, 0, None, None, np.zeros(0, np.float32))] + _params(H, [(RNN, 0, 2)], seed=n)
    toks = list(range(n))
    w, outs = c.build([toks], params, H, table)
    h = _oracle_states(w)
    P = oracle_params(w)[1]

    def direct(xs):
        if len(xs) == 1:
            return table[xs[0]].astype(np.float64)
        m = len(xs) // 2
        hh, _, _ = OC.forward_node(RNN, P, H, None, [direct(xs[:m]), direct(xs[m:])], [np.zeros(H), np.zeros(H)])
        return hh

    np.testing.assert_allclose(h[outs[0].id], direct(toks), rtol=1e-12, atol=1e-14)
    assert w.num_nodes == 2 * n - 1


def test_optional_and_errors():
    c = B.Compiler(B.Optional(B.Scalar()))
    _, out = c.trace(None)
    assert out is B.ZERO
    _, out = c.trace(3)
    assert out == B.Row(3)
    bad = B.Compiler(B.AllOf(B.Zeros(), B.Zeros()) >> B.Op(TL, 0))  # a Tree-LSTM with no input and no child
    with pytest.raises(ValueError):
        bad.trace(0)
    with pytest.raises(RuntimeError):
        B.Compiler(B.ForwardDeclaration()()).trace(0)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_compiled_trees_on_gpu(dtype):
    from tests import gpu_common as C
    rng = np.random.default_rng(7)
    H, V = 40, 200
    trees = [random_tree(rng, int(n), V) for n in rng.integers(1, 40, 64)]
    table = gen._finish_values(0.3 * rng.standard_normal((V, H)), dtype)
    params = _params(H, [(TL, H, 2)], dtype=dtype, seed=3)
    w, outs = B.Compiler(tree_lstm_expr()).build(trees, params, H, table, dtype=dtype, seed=5)
    g = C.run_device(w, table_grad=True)
    o = C.run_oracle(w, table_grad=True)
    C.compare_all(w, g, o, table_grad=True)
    ids = [out.id for out in outs]
    from oracle import compare
    assert compare.rel_err(g["h"][ids], o["h"][ids]) <= C.TOL[dtype]


SC, SM, AO, PJ = gen.KIND_ATTN_SCORE, gen.KIND_ATTN_SUM, gen.KIND_ATTN_OUT, gen.KIND_PROJ


def attention_expr():
    """Feed-forward attention over a sequence of token rows (Section 3.4): h_t = f(x_t) (embedding, PROJ f),
    scored, the scored items merged by a balanced Reduce, the attention output, then PROJ g."""
    item = B.Scalar() >> B.Op(EMB, 0) >> B.Op(PJ, 1) >> B.Op(SC, 2)
    return B.Map(item) >> B.Reduce(B.Op(SM, 3)) >> B.Op(AO, 4) >> B.Op(PJ, 5)


def _attention_params(H, dtype="f32", seed=0):
    rng = np.random.default_rng(seed)
    return [gen.ParamSet(EMB, H, 0, None, None, np.zeros(0, np.float32)),
            gen.make_param_set(rng, PJ, 0, 1, H, dtype),
            gen.make_param_set(rng, SC, 0, 1, H, dtype),
            gen.make_param_set(rng, SM, 0, 2, H, dtype),
            gen.make_param_set(rng, AO, 0, 1, H, dtype),
            gen.make_param_set(rng, PJ, 0, 1, H, dtype)]


def test_attention_expression_matches_the_softmax_equation():
    """The compiled attention model evaluated by the oracle equals g(softmax(w . f(x_t) + b) . f(x_t)) computed
    directly from the equation on each whole sequence (scipy's softmax); the empty sequence gives g(0)."""
    from scipy.special import softmax
    H, V = 6, 30
    c = B.Compiler(attention_expr())
    assert c.ops == [gen.OpSpec(EMB, 0, 1, 0), gen.OpSpec(PJ, 1, 0, 1), gen.OpSpec(SC, 1, 0, 2),
                     gen.OpSpec(SM, 2, 0, 3), gen.OpSpec(AO, 1, 0, 4), gen.OpSpec(PJ, 1, 0, 5)]
    rng = np.random.default_rng(9)
    table = rng.standard_normal((V, H)).astype(np.float32)
    params = _attention_params(H, seed=9)
    params[2].W_rec = rng.uniform(-1, 1, (H, 1)).astype(np.float32)  # peaked weights: a stronger check
    seqs = [[int(x) for x in rng.integers(0, V, n)] for n in (1, 2, 5, 16, 33)] + [[]]
    w, outs = c.build(seqs, params, H, table)
    h = _oracle_states(w)
    P = oracle_params(w)
    f = lambda x: np.tanh(x @ P[1]["W_rec"] + P[1]["bias"])
    g = lambda x: np.tanh(x @ P[5]["W_rec"] + P[5]["bias"])
    for s, out in zip(seqs, outs):
        if s:
            hs = f(table[s].astype(np.float64))
            e = hs @ P[2]["W_rec"][:, 0] + P[2]["bias"][0]
            want = g(softmax(e) @ hs)
        else:
            want = g(np.zeros(H))
        np.testing.assert_allclose(h[out.id], want, rtol=1e-12, atol=1e-14)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_compiled_attention_on_gpu(dtype):
    from tests import gpu_common as C
    rng = np.random.default_rng(8)
    H, V = 64, 300
    seqs = [[int(x) for x in rng.integers(0, V, n)] for n in rng.integers(0, 60, 48)]
    table = gen._finish_values(rng.standard_normal((V, H)), dtype)
    w, outs = B.Compiler(attention_expr()).build(seqs, _attention_params(H, dtype, seed=4), H, table, dtype=dtype,
                                                 seed=6)
    g = C.run_device(w, table_grad=True)
    C.assert_schedule_equal(g["sched"], C.oracle_schedule(w))
    o = C.run_oracle(w, table_grad=True)
    # the scorer's bias gradient is exactly 0 here (only the outputs carry a gradient and softmax ignores a
    # common shift of the scores): compared against the magnitude of its terms instead of its own value; the
    # gradient of an attention node's c (its one entry ds) as one tensor
    db = float(g["grads"][2]["bias"][0])
    g["grads"][2]["bias"] = None
    C.compare_all(w, g, o, table_grad=True, whole_keys=("dc",))
    assert abs(db - float(o["grads"][2]["bias"][0])) <= C.TOL[dtype] * C.scorer_terms(w, o, 2)
