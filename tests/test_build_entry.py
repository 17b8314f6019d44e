"""The build entry point must work in a fresh checkout, where libdv.so does
not exist yet: it may not import the package (which loads the library)
before compiling it."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_build_script_loads_without_the_library():
    code = ("import __graft_entry__ as g, sys; m = g._hip_build_module(); "
            "assert callable(m.build) and m.LIB.endswith('libdv.so'); "
            "assert 'paper_2403_06988_amd' not in sys.modules")
    env = dict(os.environ, DV_LIBRARY=os.path.join(ROOT, "no-such-dir", "libdv.so"))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_package_import_fails_loudly_without_the_library():
    env = dict(os.environ, DV_LIBRARY=os.path.join(ROOT, "no-such-dir", "libdv.so"))
    r = subprocess.run([sys.executable, "-c", "import paper_2403_06988_amd"], cwd=ROOT, env=env,
                       capture_output=True, text=True)
    assert r.returncode != 0 and "no CPU fallback" in r.stderr
