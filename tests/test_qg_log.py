"""QG_LOG: with the variable set, every status-returning entry point prints
one line (name, scalar arguments, status) to stderr; unset, nothing. The
calls fail host-side validation, so no GPU is touched."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CODE = ("import paper_2609_21849_amd as q; L = q.lib(); "
        "print(L.qg_gemm(1, None, None, None, 128, 1, None, 0, 4, 40, 128, None, 40, 0, None)); "
        "print(L.qg_quantize_act(7, None, 1, 16, 16, None, None, None, None))")


def run(env_value):
    env = dict(os.environ)
    env.pop("QG_LOG", None)
    if env_value is not None:
        env["QG_LOG"] = env_value
    return subprocess.run([sys.executable, "-c", CODE], env=env, cwd=ROOT, capture_output=True, text=True,
                          timeout=120)


def test_log_lines_when_enabled():
    r = run("1")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stderr.splitlines() if l.startswith("[qgemm]")]
    assert len(lines) == 2, r.stderr
    assert lines[0].startswith("[qgemm] qg_gemm(a_fmt=1 w_fmt=1 m=4 n=40 k=128 ") and lines[0].endswith(
        "-> shape breaks the layout contract")
    assert lines[1] == "[qgemm] qg_quantize_act(fmt=7 rows=1 cols=16 ldx=16) -> invalid argument"
    assert r.stdout.split() == ["3", "1"]


def test_silent_when_unset_or_zero():
    for v in (None, "0", ""):
        r = run(v)
        assert r.returncode == 0 and "[qgemm]" not in r.stderr, (v, r.stderr[-500:])
