"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(host code only, gcc) runs the verify, greedy, drafter-sampling and
row-statistics entry points on small workloads without a report."""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402

SCRIPT = textwrap.dedent("""
    import sys
    import numpy as np
    sys.path.insert(0, {root!r})
    sys.path.insert(0, {tests!r})
    import oracle, parity
    from paper_2405_19261_amd import workloads as W
    for cfg, kw in [(1, {{}}), (2, dict(B=2, V=3001)), (3, dict(B=2, V=5000)),
                    (5, dict(B=6, V=2000)), (3, dict(B=2, V=4000, rule=W.TOKEN_V2, alpha=0.05)),
                    (3, dict(B=2, V=4000, rule=W.OPTLOG, alpha=1.0)),
                    (3, dict(B=2, V=4000, rule=W.BILD, alpha=6.0)),
                    (3, dict(B=2, V=4000, rule=W.LOSSY, alpha=0.3))]:
        wl = W.WORKLOADS[cfg].with_(**kw)
        h = parity.host_inputs(W.generate(wl, 0, "cpu"))
        o = parity.run_oracle(h)
        assert (o["accept_len"] >= 0).all()
        g = parity.run_oracle(h, greedy=True)
        assert (g["accept_len"] >= 0).all()
        z = h["q"][:, 0]
        t = oracle.draft_sample(z, np.full(z.shape[0], 0.7, np.float32),
                                np.linspace(0.05, 0.95, z.shape[0]).astype(np.float32))
        assert (np.asarray(t[0] if isinstance(t, tuple) else t) >= 0).all()
        oracle.softmax_row(z[0], 0.5)
    print("sanitized oracle ok")
""")


def test_oracle_under_asan_ubsan(tmp_path):
    libasan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    if not os.path.isabs(libasan) or not os.path.exists(libasan):
        pytest.skip("libasan not available")
    lib = str(tmp_path / "libspc_oracle_san.so")
    oracle.build(out=lib, extra=["-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                                       "-fno-sanitize-recover=all", "-O1"])
    env = dict(os.environ)
    env["SPC_ORACLE_LIB"] = lib
    # the sanitizer runtime must come first among the preloaded libraries
    env["LD_PRELOAD"] = ":".join(x for x in (libasan, os.environ.get("LD_PRELOAD", "")) if x)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:exitcode=23"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1:exitcode=24"
    env["OMP_NUM_THREADS"] = "2"
    code = SCRIPT.format(root=ROOT, tests=os.path.join(ROOT, "tests"))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600)
    report = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, report
    assert "sanitized oracle ok" in r.stdout, report
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, report
