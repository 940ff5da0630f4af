"""Planted mistakes in the oracle must fail its pins.

Each case copies the oracle into a temporary directory, plants one plausible
mistake (a dropped term, a wrong coefficient, sign or index, a swapped
operand), and runs the pin suite against the copy in a subprocess.  The pin
suite must fail for every mistake.  CPU only; the real oracle is untouched.
"""
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PIN_FILES = ("test_oracle_pins.py", "test_oracle_variants.py")

# (file, original text, planted mistake, what it breaks)
MUTATIONS = [
    ("dsm_oracle.py", "m_new = beta1_ * m + one_minus_b1 * g",
     "m_new = beta1_ * m + one_minus_b2 * g", "AdamW first-moment coefficient"),
    ("dsm_oracle.py", "\n    m_hat = m_new / bc1", "\n    m_hat = m_new", "AdamW bias correction dropped"),
    ("dsm_oracle.py", "(m_hat / (np.sqrt(v_hat) + eps_) + wd_ * x)",
     "(m_hat / np.sqrt(v_hat + eps_) + wd_ * x)", "AdamW epsilon placement"),
    ("dsm_oracle.py", "x_new = x - lr_ * (m_hat", "x_new = x + lr_ * (m_hat", "AdamW step sign"),
    ("dsm_oracle.py", "+ wd_ * x)", "+ wd_ * m_hat)", "AdamW decay operand"),
    ("dsm_oracle.py", "m_new = mu * m + g", "m_new = mu * m + (1 - mu) * g",
     "Polyak momentum dampened"),
    ("dsm_oracle.py", "u = beta1_ * mp + c1 * delta", "u = beta2_ * mp + c1 * delta",
     "u uses beta2"),
    ("dsm_oracle.py", "m_new = beta2_ * mp + c2 * delta", "m_new = beta2_ * mp + c1 * delta",
     "momentum uses (1-beta1)"),
    ("dsm_oracle.py", "u = beta1_ * mp + c1 * delta",
     "u = beta1_ * (beta2_ * mp + c2 * delta) + c1 * delta", "u from the new momentum"),
    ("dsm_oracle.py", "x_new = xp - step * (S + lam_p * xp)", "x_new = xp - step * S",
     "global weight decay dropped"),
    ("dsm_oracle.py", "lam_p = lam_ if decay[p] else dt(0.0)\n        # Eq. (7)",
     "lam_p = lam_\n        # Eq. (7)", "decay mask ignored"),
    ("dsm_oracle.py", "\n        m_hat = m_new / bc1", "\n        m_hat = m_new",
     "Global AdamW bias correction dropped"),
    ("dsm_oracle.py", "for i in range(1, n):", "for i in range(1, n - 1):",
     "last worker dropped from the average"),
    ("dsm_oracle.py", "delta = acc / dt(n)", "delta = acc", "average not divided by n"),
    ("dsm_oracle.py", "c1 = dt((1.0 - b1) / g_)", "c1 = dt((1.0 - b1) * g_)",
     "1/gamma scaling inverted"),
    ("dsm_oracle.py", "step = dt(f32(eta) * g_)", "step = dt(f32(eta))",
     "global step not scaled by gamma"),
    ("dsm_oracle.py", "return np.sign(u) + u.dtype.type(0.0)",
     "return np.where(u >= 0, 1.0, -1.0).astype(u.dtype)", "sign(0) taken as +1"),
    ("dsm_oracle.py", "keep = _exact_less(2 * k - (1 << 24), B, au)",
     "keep = _exact_less(k, B, au)", "Eq. (9) threshold replaced by Eq. (10)'s"),
    ("dsm_oracle.py", "return np.where(keep, s, dt(0.0) - s)",
     "return np.where(keep, s, s)", "Eq. (9) never flips"),
    ("dsm_oracle.py", "B = np.max(np.abs(u)) if u.size else dt(0.0)",
     "B = np.max(u) if u.size else dt(0.0)", "bound without absolute value"),
    ("dsm_oracle.py", "w = philox4x32_10(q, tensor_index, t, PHILOX_STREAM,",
     "w = philox4x32_10(q, t, tensor_index, PHILOX_STREAM,", "Philox counter words swapped"),
    ("philox.py", "n0 = (p1 >> sh) ^ c1 ^ np.uint64(k0)",
     "n0 = (p1 >> sh) ^ c1 ^ np.uint64(k1)", "Philox key word swapped"),
    ("philox.py", "        p0 = M0 * c0\n", "        p0 = M1 * c0\n", "Philox multiplier swapped"),
    ("dsm_oracle.py", '    st["replicas"] = synchronize(st["x"], st["n"])',
     '    st["replicas"] = synchronize(st["x"], st["n"]) if False else st["replicas"]',
     "replicas not synchronised"),
    ("dsm_oracle.py", "u = beta1_ * mp + c1 * sign(delta)", "u = beta1_ * mp + c1 * delta",
     "signed SlowMo without the sign"),
    ("dsm_oracle.py", "out[\"x\"].append(xp - step * (u + lam_p * xp))",
     "out[\"x\"].append(xp - step * (sign(u) + lam_p * xp))", "Lookahead keeps the sign"),
    ("dsm_oracle.py", "g = inv_gamma * delta", "g = delta", "Global AdamW without 1/gamma"),
    ("dsm_oracle.py", "bc1 = dt(1.0 - beta_power(b1, t + 1))", "bc1 = dt(1.0 - beta_power(b1, t + 2))",
     "Global AdamW bias correction off by one"),
    ("dsm_oracle.py", "x_new = xp - eta_ * (m_hat", "x_new = xp - eta_ * inv_gamma * (m_hat",
     "Global AdamW step scaled by 1/gamma"),
    ("dsm_oracle.py",
     "    local_steps(st, grads, H=H, decay=decay, first_step=t * H + 1, prec=prec, **local)",
     "    st['s1'] = [[a * 0 for a in w] for w in st['s1']]\n"
     "    local_steps(st, grads, H=H, decay=decay, first_step=t * H + 1, prec=prec, **local)",
     "worker momentum reset every round"),
    ("dsm_oracle.py", "close = (np.isfinite(lhs) & np.isfinite(rhs) &",
     "close = (np.ones_like(res) &", "exact re-check applied to infinite sides"),
    ("dsm_oracle.py", "res = lhs < rhs", "res = ~(lhs >= rhs)",
     "a NaN comparison keeps the sign"),
    ("dsm_oracle.py", "first_step=t * H + 1, prec=prec, **local)",
     "first_step=1, prec=prec, **local)", "bias-correction count restarted every round"),
    ("dsm_oracle.py",
     "    local_steps(st, grads, H=H, decay=decay, first_step=t * H + 1, prec=prec, **local)",
     "    if st['s2'] is not None:\n"
     "        st['s2'] = [[a * 0 for a in w] for w in st['s2']]\n"
     "    local_steps(st, grads, H=H, decay=decay, first_step=t * H + 1, prec=prec, **local)",
     "AdamW second moment reset every round"),
    ("dsm_oracle.py", "\n    v_hat = v_new / bc2", "\n    v_hat = v_new / bc1",
     "AdamW second moment divided by the first moment's bias correction"),
    ("dsm_oracle.py", "t=t, prec=prec, **glob, **extra)", "t=0, prec=prec, **glob, **extra)",
     "round driver passes t = 0 to every global step"),
    ("dsm_oracle.py", "        lam_p = lam_ if decay[p] else dt(0.0)\n        x_new = xp - eta_",
     "        lam_p = lam_\n        x_new = xp - eta_", "Global AdamW ignores the decay mask"),
    ("dsm_oracle.py", "        keep = _exact_less(2 * k - (1 << 24), B, au)",
     "        keep = _exact_less(2 * k - (1 << 24) + 1, B, au)", "Eq. (9) threshold one count off"),
    ("dsm_oracle.py", "    B = float(B)\n", "    B = float(B) * (1 + 2.0 ** -40)\n",
     "randomized decision not exact (bound off by 2^-40)"),
    ("dsm_oracle.py", "    if not np.isfinite(B):\n        return np.full(",
     "    if np.isnan(B):\n        return np.full(",
     "an infinite bound decided by the limit of the probabilities"),
    ("dsm_oracle.py", "    if not np.isfinite(B):\n        return np.full(",
     "    if False:\n        return np.full(",
     "a non-finite bound decided by bare IEEE comparisons (reversed or frozen tensor)"),
]


def _run_mutant(case):
    fname, orig, planted, _ = case
    tmp = tempfile.mkdtemp(prefix="dsm_mut_")
    try:
        shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(tmp, "oracle"),
                        ignore=shutil.ignore_patterns("__pycache__"))
        tdir = os.path.join(tmp, "tests")
        os.makedirs(tdir)
        for f in PIN_FILES:
            shutil.copy(os.path.join(HERE, f), tdir)
        shutil.copytree(os.path.join(HERE, "golden"), os.path.join(tdir, "golden"))
        shutil.copytree(os.path.join(HERE, "native"), os.path.join(tdir, "native"),
                        ignore=shutil.ignore_patterns("bin"))
        with open(os.path.join(tdir, "conftest.py"), "w") as f:
            f.write("import os, sys\nsys.path.insert(0, os.path.dirname(os.path.dirname("
                    "os.path.abspath(__file__))))\n")
        path = os.path.join(tmp, "oracle", fname)
        src = open(path).read()
        assert src.count(orig) == 1, f"mutation anchor not unique: {orig!r}"
        open(path, "w").write(src.replace(orig, planted))
        env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            *[os.path.join(tdir, f) for f in PIN_FILES]],
                           cwd=tmp, env=env, capture_output=True, text=True, timeout=600)
        return r.returncode, r.stdout[-2000:]
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


def test_every_planted_mistake_fails_a_pin():
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(_run_mutant, MUTATIONS))
    survivors = [(case[3], out) for case, (rc, out) in zip(MUTATIONS, results) if rc == 0]
    errors = [(case[3], out) for case, (rc, out) in zip(MUTATIONS, results)
              if rc not in (0, 1)]
    assert not errors, f"pin suite errored instead of failing: {errors}"
    assert not survivors, "mutants not caught: " + ", ".join(s for s, _ in survivors)


def test_unmutated_copy_passes():
    """Control: the same harness with an unchanged oracle passes."""
    rc, out = _run_mutant(("dsm_oracle.py", "PHILOX_STREAM = 1", "PHILOX_STREAM = 1", "none"))
    assert rc == 0, out
