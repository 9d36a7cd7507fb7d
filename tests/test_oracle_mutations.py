"""Planted mistakes in a copy of the oracle must fail its pins.

Each case copies oracle/ to a temporary directory, applies one textual mutation
(a dropped term, a wrong sign, a wrong index, a transposed operand, a flipped
comparison, a dropped filter), builds it, and runs tests/test_oracle_pins.py against the copy in a
subprocess.  The pins must fail.  This runs on the CPU only.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")

MUTATIONS = [
    # (file, original text, planted mistake)
    ("cospec_oracle.c", "if (x > m) {", "if (x >= m) {"),                       # ties to the last index
    ("cospec_oracle.c", "h -= exp(logp) * logp;", "h += exp(logp) * logp;"),    # entropy sign
    ("cospec_oracle.c", "double lse = m + log(s);", "double lse = log(s);"),   # dropped max shift
    ("cospec_oracle.c", "s += exp(oracle_elem(row, dtype, v) - m);",
     "s += exp(oracle_elem(row, dtype, v) - m) * (v > 0);"),                    # dropped first term
    ("cospec_oracle.c", "double r = u > 0.0 ? u : 0.0;", "double r = u;"),     # dropped ReLU
    ("cospec_oracle.c", "double u = b1 ? oracle_elem(b1, dtype, j) : 0.0;", "double u = 0.0;"),
    ("cospec_oracle.c", "oracle_elem(w1, dtype, j * d + c)", "oracle_elem(w1, dtype, c * hdim + j)"),
    ("cospec_oracle.c", "double z = b2;", "double z = 0.0;"),                  # dropped b2
    ("__init__.py", "if not delta[i - 1] and not accept[i - 1]]", "if not delta[i - 1] and accept[i - 1]]"),
    ("__init__.py", "[int(target_argmax[s - 1])]", "[int(target_argmax[s])]"),   # wrong emitted row
    ("__init__.py", "ytil = cand[:, :K]", "ytil = cand[:, 1:]"),                # verify against wrong row
    ("__init__.py", "ytil = cand[:, :K]", "ytil = ts.arg[:, :K]"),              # T = 1 sample ignored
    ("__init__.py", "tokens[b] = chain_tokens(s, toks[b], cand[b])",
     "tokens[b] = chain_tokens(s, toks[b], ts.arg[b])"),                        # emits the argmax at T = 1
    ("cospec_oracle.c", "p[v] = exp(oracle_elem(row, dtype, v) - lse);",
     "p[v] = exp(oracle_elem(row, dtype, v));"),                                # unnormalised probabilities
    ("cospec_oracle.c", "if (at > u[r]) {\n                pick = v;",
     "if (at > u[r]) {\n                pick = v + 1 < V ? v + 1 : v;"),         # one past the crossing
    ("cospec_oracle.c", "at = before + work[v];", "at = work[v];"),              # not cumulative
    ("__init__.py", "if i <= min(s, K):", "if i < min(s, K):"),                  # drops the stopping decision
    ("__init__.py", "rho = (s - i_star) / ((K + 1) - i_star)", "rho = (s - i_star) / (K - i_star + 1e-9)"),
    ("__init__.py", "s_acc[i - 1] = bool(accept[i - 1]) and i < i_rej",
     "s_acc[i - 1] = i <= i_rej"),                                            # rejected one in S_acc
    ("__init__.py", "- beta * s_rej[i - 1])", "+ beta * s_rej[i - 1])"),        # rejection rewarded
    ("__init__.py", "accept = u < pi", "accept = u <= pi"),
    ("cospec_oracle.c", "p[v] = p[v] > q[v] ? p[v] - q[v] : 0.0;", "p[v] = p[v] - q[v];"),   # unclipped residual
    ("__init__.py", "accept = uu[:, :K] < ratio", "accept = uu[:, :K] < 1.0 / ratio"),        # inverted ratio
    ("__init__.py", "vis = np.arange(p + 1) if p < lc else np.arange(ln)",
     "vis = np.arange(p + 1) if p <= lc else np.arange(ln)"),                  # first SEP causal
    ("__init__.py", "                    out[b, i, j] = j <= i\n", "                    out[b, i, j] = j < i + 2\n"),
    ("__init__.py", "kh = h // grp", "kh = h % Hkv"),                             # wrong query-head group
    ("__init__.py", "t = target_seq[s - 1: s]", "t = target_seq[s - 2: s - 1]"),           # resample wrong row
    ("__init__.py", "logp_tgt = _gather(target[:, :K, :], toks)", "logp_tgt = _gather(target[:, 1:, :], toks)"),
    ("__init__.py", "if ok[n] and depth[n] > depth[best]:", "if ok[n] and depth[n] >= depth[best]:"),
    ("__init__.py", "accept = pi > lam", "accept = pi >= lam"),                # non-strict threshold
    ("__init__.py", "ok[n] = ok[p] and bool(passed[n])", "ok[n] = bool(passed[n])"),  # ignores ancestors
    ("__init__.py", "if not delta[n] and ambiguous[n] and not blocked[int(parent[n])]]",
     "if not delta[n] and not blocked[int(parent[n])]]"),                       # certain decisions set free
    ("__init__.py", "blocked[n] = blocked[p] or certain_fail", "blocked[n] = certain_fail"),  # not inherited
    ("__init__.py", "free = [i for i in range(limit) if not delta[i] and ambiguous[i]]",
     "free = [i for i in range(limit) if not delta[i]]"),                       # chain: certain set free
    ("cospec_oracle.c", "out_lo[r] = before / z;", "out_lo[r] = before;"),     # residual not normalised
    ("cospec_oracle.c", "out_hi[r] = (before + p[pick]) / z;", "out_hi[r] = (before + p[pick + 1]) / z;"),
    ("cospec_oracle.c", "before += p[v];\n        out_lo[r]", "before += p[v] + p[pick];\n        out_lo[r]"),
]


@pytest.mark.parametrize("fname,old,new", MUTATIONS, ids=[f"{m[0]}:{m[2][:40]}" for m in MUTATIONS])
def test_planted_mistake_fails_pins(tmp_path, fname, old, new):
    dst = tmp_path / "oracle_mut"
    dst.mkdir()
    for f in ("__init__.py", "cospec_oracle.c"):
        shutil.copy(os.path.join(ORACLE, f), dst / f)
    text = (dst / fname).read_text()
    assert text.count(old) == 1, f"mutation anchor not found once: {old!r}"
    (dst / fname).write_text(text.replace(old, new))
    env = dict(os.environ, COSPEC_ORACLE_UNDER_TEST=str(dst))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 1, f"pins did not catch {new!r}:\n{r.stdout[-2000:]}"
