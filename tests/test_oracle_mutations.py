"""The oracle's pins must reject plausible mistakes in the oracle.

Each case copies the oracle package to a temporary directory, plants one
mistake in the copy (a dropped term, a wrong sign, a wrong index, a transposed
operand, multiplying by the temperature), and runs the pin tests against the
copy; they must fail. The real oracle files are never modified.
"""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = [
    ("logprobs.py", "z /= float(temperature)", "z *= float(temperature)"),
    ("logprobs.py", "ent[r0:r1] = -(p * zc).sum(axis=1)", "ent[r0:r1] = (p * zc).sum(axis=1)"),
    ("logprobs.py", "ent[r0:r1] = -(p * zc).sum(axis=1)", "ent[r0:r1] = -(p * (z - m)).sum(axis=1)"),
    ("logprobs.py", "lp[ok] = zc[rows[ok], tok[ok]]", "lp[ok] = zc[rows[ok], np.minimum(tok[ok] + 1, V - 1)]"),
    ("logprobs.py", "lse = m + np.log(", "lse = 0 * m + np.log("),
    ("logprobs.py", "np.exp(z - m).sum(axis=1, keepdims=True)", "np.exp(z - m)[:, 1:].sum(axis=1, keepdims=True)"),
    ("logprobs.py", "h @ bf16_to_f64(w_bits[v0:v1]).T", "h[:, ::-1] @ bf16_to_f64(w_bits[v0:v1]).T"),
    ("logprobs.py", "<< np.uint32(16)", "<< np.uint32(15)"),
    ("mismatch.py", "delta = a - b", "delta = b - a"),
    ("mismatch.py", "k3 = np.expm1(delta) - delta", "k3 = np.expm1(delta) + delta"),
    ("mismatch.py", "k3 = np.expm1(delta) - delta", "k3 = np.exp(delta) - delta"),
    ("mismatch.py", "w = np.minimum(np.exp(delta), float(C))", "w = np.maximum(np.exp(delta), float(C))"),
    ("mismatch.py", "w = np.minimum(np.exp(delta), float(C))", "w = np.minimum(np.exp(-delta), float(C))"),
    ("mismatch.py", "per_token = -delta if", "per_token = delta if"),
    ("mismatch.py", "score[j] = math.fsum(per_token[s0:s1].tolist())", "score[j] = math.fsum(per_token[s0:s1 + 1].tolist())"),
    ("mismatch.py", "keep[j] = bool(score[j] <= tau_seq)", "keep[j] = bool(score[j] < tau_seq)"),
    ("mismatch.py", "        if keep[j]:\n", "        if True:\n"),
    ("mismatch.py", "else np.expm1(delta) - delta\n", "else np.expm1(delta) + delta\n"),
    ("grads.py", "* p * (q + H)", "* p * (q - H)"),
    ("grads.py", "* (onehot - p) - e[r0:r1, None]", "* (onehot - p) + e[r0:r1, None]"),
    ("grads.py", "gb * (onehot - p)", "gb * onehot"),
    ("grads.py", "dacc[r0:r1] = dz / float(temperature)", "dacc[r0:r1] = dz * float(temperature)"),
    ("grads.py", "onehot[rows[ok], tok[ok]] = 1.0", "onehot[rows[ok], np.minimum(tok[ok] + 1, V - 1)] = 1.0"),
    ("grads.py", "gb = np.where(ok, g[r0:r1], 0.0)", "gb = g[r0:r1]"),
    ("grads.py", "dw = dacc.T @ h", "dw = dacc.T @ h[::-1]"),
    ("grads.py", "dh = dacc @ w", "dh = dacc @ w[::-1]"),
    ("rmsnorm.py", "np.rint(m * 256.0)", "np.floor(m * 256.0 + 0.5)"),
    ("rmsnorm.py", "np.rint(m * 256.0) / 256.0", "np.rint(m * 128.0) / 128.0"),
    ("rmsnorm.py", "(x * x).sum(axis=1) / d + float(eps))", "(x * x).sum(axis=1) + float(eps))"),
    ("rmsnorm.py", "[None, :] * h)", "[None, :] * n)"),
    ("rmsnorm.py", "G - (r ** 3 * s / d)", "G + (r ** 3 * s / d)"),
    ("rmsnorm.py", "(r ** 3 * s / d)", "(r ** 2 * s / d)"),
    ("rmsnorm.py", "s = (G * g[None, :] * x)", "s = (G * x)"),
    ("rmsnorm.py", "dg = (G * x * r[:, None])", "dg = (G * x)"),
    ("ppo.py", "r = np.exp(lp - lo)", "r = np.exp(lo - lp)"),
    ("ppo.py", "L = -np.minimum(unclipped, clipped_term)", "L = -np.maximum(unclipped, clipped_term)"),
    ("ppo.py", "np.clip(r, 1.0 - eps_low, 1.0 + eps_high)", "np.clip(r, 1.0 - eps_high, 1.0 + eps_low)"),
    ("ppo.py", "np.where(use_unclipped, -A * r, 0.0)", "np.where(use_unclipped, -A, 0.0)"),
    ("ppo.py", "grad_tok[s0:s1] / n", "grad_tok[s0:s1]"),
    ("ppo.py", "C = -(r - 1.0) * A", "C = (r - 1.0) * A"),
    ("ppo.py", "token_loss[s0:s1] = w[s0:s1] * L[s0:s1]", "token_loss[s0:s1] = L[s0:s1]"),
    ("ppo.py", "math.fsum(seq.tolist()) / n", "math.fsum(seq.tolist()) / T"),
    ("ppo.py", "use_unclipped = unclipped <= clipped_term", "use_unclipped = unclipped >= clipped_term"),
]


@pytest.mark.parametrize("fname,old,new", MUTATIONS, ids=[m[2][:40] for m in MUTATIONS])
def test_pins_reject_planted_mistake(tmp_path, fname, old, new):
    dst = tmp_path / "oracle"
    shutil.copytree(os.path.join(ROOT, "oracle"), dst, ignore=shutil.ignore_patterns("__pycache__"))
    text = (dst / fname).read_text()
    assert old in text, f"mutation anchor not found in oracle/{fname}: {old!r}"
    (dst / fname).write_text(text.replace(old, new, 1))
    env = dict(os.environ)
    env["PYTHONPATH"] = os.pathsep.join([str(tmp_path), ROOT])
    env["PYTHONDONTWRITEBYTECODE"] = "1"
    code = ("import sys; sys.path.insert(0, %r); import oracle; "
            "assert oracle.__file__.startswith(%r), oracle.__file__; "
            "import pytest; sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', %r]))"
            % (str(tmp_path), str(tmp_path), os.path.join(ROOT, "tests", "test_oracle.py")))
    r = subprocess.run([sys.executable, "-c", code], cwd=str(tmp_path), env=env,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"pins did not catch: {new!r}\n{r.stdout[-2000:]}"
    assert "passed" in r.stdout or "failed" in r.stdout, r.stdout[-2000:] + r.stderr[-2000:]
