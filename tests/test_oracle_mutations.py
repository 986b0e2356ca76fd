"""Plants plausible mistakes in a scratch copy of the oracle (on the CPU) and checks
that the oracle's pins catch every one of them: a wrong gate, a wrong weight
block, a dropped bias, swapped gate columns, a sign flip, swapped child
gradients, a dropped upstream term, a scaled weight gradient, a wrong tanh
derivative, a lost cell-state pass-through, wrong sort keys and tie-breaks,
min instead of max in the depth rule, node ids instead of positions as edge
labels, overwriting instead of summing fan-out contributions, and in the parity metric: the per-row
floor dropped, min instead of max over rows, the row norm taken as a min, whole= ignored, rows cut along
the last axis, and NaN rows skipped; in the paper-form schedule: pass-throughs numbered among the user
operations, a pass-through one depth too early, labels into the reader's own depth, and a concatenation
taken row by row instead of output slot by output slot; in feed-forward attention: the merge exponent's
sign flipped, min instead of max as the running maximum, the scorer's bias dropped, the score gradient's
cell-state term dropped, the pass-through term of the scored item's gradient dropped, an unscaled sum
gradient, and the output's normaliser gradient with the wrong sign."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = [
    ("cells.py", "c = i * um + fl * cl + fr * cr", "c = i * um + fl * cl + fl * cr"),
    ("cells.py", 'z += h @ P["W_rec"][k * H:(k + 1) * H]', 'z += h @ P["W_rec"][0:H]'),
    ("cells.py", 'z = np.array(P["bias"], dtype=np.float64, copy=True)',
     'z = 0 * np.array(P["bias"], dtype=np.float64, copy=True)'),
    ("cells.py", "o = sigmoid(z[2 * H:3 * H])\n        u = np.tanh(z[3 * H:4 * H])",
     "u = np.tanh(z[2 * H:3 * H])\n        o = sigmoid(z[3 * H:4 * H])"),
    ("cells.py", "            dh * tc * o * (1.0 - o),\n            dct * i * m * (1.0 - u * u),\n        ])\n        dcs = [dct * fl, dct * fr]",
     "            -dh * tc * o * (1.0 - o),\n            dct * i * m * (1.0 - u * u),\n        ])\n        dcs = [dct * fl, dct * fr]"),
    ("cells.py", "dcs = [dct * fl, dct * fr]", "dcs = [dct * fr, dct * fl]"),
    ("cells.py", "dct = dc + dh * o * (1.0 - tc * tc)\n        dz = np.concatenate([\n            dct * (m * u) * i * (1.0 - i),\n            dct * cl",
     "dct = dh * o * (1.0 - tc * tc)\n        dz = np.concatenate([\n            dct * (m * u) * i * (1.0 - i),\n            dct * cl"),
    ("cells.py", 'grads["W_in"] = np.outer(x, dz)', 'grads["W_in"] = np.outer(x, dz) * (1 + 1e-3)'),
    ("cells.py", "dz = dh * (1.0 - h * h)", "dz = dh * (1.0 - h)"),
    ("cells.py", "dcs = [np.array(dc, dtype=np.float64)] if kind == PROJ", "dcs = [np.zeros(H)] if kind == PROJ"),
    ("schedule.py", "return (depth[v] - 1) * num_ops + int(node_op[v])",
     "return int(node_op[v]) * 100000 + depth[v]"),
    ("schedule.py", "key=lambda v: (key(v), v)", "key=lambda v: (key(v), -v)"),
    ("schedule.py", "d = max(d, depth[c])", "d = min(d, depth[c]) if d else depth[c]"),
    ("schedule.py", "child_pos.append(node_pos[c] if c >= 0 else -1)", "child_pos.append(c if c >= 0 else -1)"),
    ("evaluate.py", "dh[k] += dhs[j]", "dh[k] = dhs[j]"),
    ("evaluate.py", 'd_table[int(batch["node_input"][v])] += dx', 'd_table[int(batch["node_input"][v])] = dx'),
    ("compare.py", "row_ref = np.maximum(np.abs(R).max(axis=1), 1e-3 * scale)", "row_ref = np.abs(R).max(axis=1)"),
    ("compare.py", "return float((np.abs(T - R).max(axis=1) / row_ref).max())",
     "return float((np.abs(T - R).max(axis=1) / row_ref).min())"),
    ("compare.py", "row_ref = np.maximum(np.abs(R).max(axis=1), 1e-3 * scale)",
     "row_ref = np.maximum(np.abs(R).min(axis=1), 1e-3 * scale)"),
    ("compare.py", "if whole or R.ndim == 1:", "if R.ndim == 1:"),
    ("compare.py", "T = T.reshape(R.shape[0], -1)\n        R = R.reshape(R.shape[0], -1)",
     "T = T.reshape(-1, R.shape[-1])\n        R = R.reshape(-1, R.shape[-1])"),
    ("compare.py", "return float((np.abs(T - R).max(axis=1) / row_ref).max())",
     "return float(np.nanmax(np.abs(T - R).max(axis=1) / row_ref))"),
    ("paper_schedule.py", "items.append((d, K + t, (1, u, k)", "items.append((d, t, (1, u, k)"),
    ("paper_schedule.py", "for d in range(depth[u] + 1, last.get((u, k), 0))",
     "for d in range(depth[u], last.get((u, k), 0))"),
    ("paper_schedule.py", "src_d = d - 1", "src_d = d"),
    ("paper_schedule.py", "        for slot, t in enumerate(its[0][4]):\n            for it in its:",
     "        for it in its:\n            for slot, t in enumerate(its[0][4]):"),
    ("cells.py", "x = [np.exp(cs[k][0] - m) if k in live", "x = [np.exp(m - cs[k][0]) if k in live"),
    ("cells.py", "m = max(cs[k][0] for k in live)", "m = min(cs[k][0] for k in live)"),
    ("cells.py", 'e = float(hc @ P["W_rec"][:, 0] + P["bias"][0])', 'e = float(hc @ P["W_rec"][:, 0])'),
    ("cells.py", "de = float(dh @ hc) + float(dc[1])", "de = float(dh @ hc)"),
    ("cells.py", "return [dh + de * w], [np.zeros(H)]", "return [de * w], [np.zeros(H)]"),
    ("cells.py", "d[1] = x[k] * dc[1]", "d[1] = dc[1]"),
    ("cells.py", "d[1] = -float(dh @ acc) / (s * s)", "d[1] = float(dh @ acc) / (s * s)"),
]


@pytest.mark.parametrize("i", range(len(MUTATIONS)))
def test_planted_mistake_is_caught(i, tmp_path):
    fname, old, new = MUTATIONS[i]
    for d in ("oracle", "tests", "paper_1702_02181_amd"):
        shutil.copytree(os.path.join(ROOT, d), tmp_path / d,
                        ignore=shutil.ignore_patterns("*.so", "__pycache__", "_build", "*.o"))
    shutil.copy(os.path.join(ROOT, "pytest.ini"), tmp_path)
    p = tmp_path / "oracle" / fname
    src = p.read_text()
    assert old in src, "mutation site moved; update the table"
    p.write_text(src.replace(old, new, 1))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:randomly",
                        "tests/test_oracle_schedule.py", "tests/test_oracle_cells.py",
                        "tests/test_oracle_compare.py", "tests/test_oracle_paper_schedule.py",
                        "tests/test_oracle_attention.py"],
                       cwd=tmp_path, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"pins missed mutation {i}: {new!r}"
