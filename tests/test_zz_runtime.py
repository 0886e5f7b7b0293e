"""The binding shares the host process's HIP runtime (torch's), never a second copy."""
import subprocess
import sys


def test_single_hip_runtime_when_binding_imported_first():
    code = ("import paper_2608_29291_amd, torch\n"
            "maps = open('/proc/self/maps').read()\n"
            "libs = {l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l}\n"
            "print(len(libs)); assert len(libs) == 1, libs\n")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       cwd=__import__("os").path.dirname(__import__("os").path.dirname(__file__)))
    assert r.returncode == 0, r.stdout + r.stderr
