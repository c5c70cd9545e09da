"""Mutation check of the oracle's pins (CPU only, not collected by pytest).

Plants one mistake at a time in a temporary copy of oracle/dqt_oracle.py (a
changed constant, a dropped term, a flipped sign, a wrong rounding or clip)
and runs the oracle's CPU tests against it; every planted mistake should make
them fail.  The repository itself is never modified.

    python tests/oracle_mutations.py
"""
import os
import shutil
import subprocess
import sys
import tempfile

# (text in the oracle, the planted mistake)
MUT = [
 ("qmax_act = np.float32(127.0)", "qmax_act = np.float32(126.0)"),
 ("pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))", "pick_hi = (d_hi <= d_lo)"),
 ("packed |= codes[:, :, j] << (2 * j)", "packed |= codes[:, :, 3 - j] << (2 * j)"),
 ("out[:, :, j] = ((packed >> (2 * j)) & 3) - 1", "out[:, :, j] = ((packed >> (2 * j)) & 3) - 2"),
 ("sq = (X * X).astype(np.float32)", "sq = (X * np.abs(X)).astype(np.float32)"),
 ("keys[~finite] = np.uint32(0xFFFFFFFF)", "keys[~finite] = np.uint32(0)"),
 ("k = int(np.floor(np.float64(np.float32(frac)) * n))", "k = int(np.ceil(np.float64(np.float32(frac)) * n))"),
 ("wp = (w - u).astype(np.float32)", "wp = (w + u).astype(np.float32)"),
 ("Xq = np.clip(np.rint(scaled), -128, 127)", "Xq = np.clip(np.floor(scaled), -128, 127)"),
 ("g[m] = max(row_max, ACT_EPS)", "g[m] = max(row_max, ACT_EPS) * np.float32(1.0000001)"),
 ("f = (np.asarray(d, dtype=np.float32) * np.float32(alpha)).astype(np.float32)", "f = (np.asarray(d, dtype=np.float32)).astype(np.float32)"),
 ("acc = a @ w.T", "acc = a @ w.T + (a[:, :1] != 0)"),
 ("dX64 = float(alpha) * (dY @ w)", "dX64 = (dY @ w)"),
 ("dW64 = dY.T @ xt_vals", "dW64 = -(dY.T @ xt_vals)"),
 ("PHILOX_M0 = 0xD2511F53", "PHILOX_M0 = 0xD2511F55"),
 ("PHILOX_W1 = 0xBB67AE85", "PHILOX_W1 = 0xBB67AE86"),
 ("return np.float32(np.float32(lr) / np.float32(alpha))", "return np.float32(np.float32(lr) * np.float32(alpha))"),
 ("delta32 = -(c * np.where(finite, g, np.float32(0))).astype(np.float32)", "delta32 = (c * np.where(finite, g, np.float32(0))).astype(np.float32)"),
 ("thresh = np.ceil(p * 2.0 ** 32)", "thresh = np.floor(p * 2.0 ** 31)"),
 ("event = U < thresh", "event = U <= thresh"),
 ("move = base + np.where(event, np.where(up_side, 1.0, -1.0), 0.0)", "move = base + np.where(event, 1.0, 0.0)"),
 ("return np.clip(x_new, qmin, qmax).astype(np.int64)", "return np.clip(x_new, qmin, qmax - 1).astype(np.int64)"),
 ("v1 = (k[\"b2\"] * v).astype(f32) + ((k[\"ob2\"] * g).astype(f32) * g).astype(f32)", "v1 = (k[\"b2\"] * v).astype(f32) + ((k[\"ob1\"] * g).astype(f32) * g).astype(f32)"),
 ("den = (np.sqrt(v1.astype(f32)) * k[\"k2\"]).astype(f32) + k[\"eps\"]", "den = (np.sqrt(v1.astype(f32)) * k[\"k2\"]).astype(f32)"),
 ("delta = -((k[\"cu\"] * u).astype(f32) + (k[\"cd\"] * q).astype(f32)).astype(f32)", "delta = -((k[\"cu\"] * u).astype(f32) - (k[\"cd\"] * q).astype(f32)).astype(f32)"),
]
src = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
tmp = tempfile.mkdtemp()
dst = os.path.join(tmp, "r")
shutil.copytree(src, dst, ignore=shutil.ignore_patterns(".git", "_work", "gpurun_out", "__pycache__", "_build"))
orig = open(os.path.join(dst, "oracle/dqt_oracle.py")).read()
tests = sorted(f"tests/{f}" for f in os.listdir(os.path.join(dst, "tests")) if f.startswith("test_oracle") or f == "test_model_cpu.py")
survived = 0
for a, b in MUT:
    assert orig.count(a) == 1, a
    open(os.path.join(dst, "oracle/dqt_oracle.py"), "w").write(orig.replace(a, b))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider", *tests],
                       cwd=dst, capture_output=True, text=True, timeout=900)
    survived += r.returncode == 0
    print("caught  " if r.returncode != 0 else "SURVIVED", a[:70], flush=True)
open(os.path.join(dst, "oracle/dqt_oracle.py"), "w").write(orig)
shutil.rmtree(tmp)
print(f"{len(MUT) - survived} of {len(MUT)} planted mistakes caught")
sys.exit(1 if survived else 0)
