"""The seeds of the seeded GPU sweeps do not depend on the process: the same
test ID draws the same inputs on every run, under any PYTHONHASHSEED, so a
failing case can be replayed from its ID."""
import os
import subprocess
import sys

from gpu_util import stable_seed

HERE = os.path.dirname(os.path.abspath(__file__))


def test_seed_of_a_fixed_id_is_a_fixed_number():
    # CRC-32 (the zlib polynomial) of the ASCII bytes of the ID
    assert stable_seed("L1N8K2C4R0S3m0p0") == 3346935489
    assert stable_seed("") == 0


def test_seeds_agree_across_hash_salts():
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from test_gpu_random_configs import CASES, case_id\n"
            "from gpu_util import stable_seed\n"
            "print(','.join(str(stable_seed(case_id(c))) for c in CASES[:10]))\n") % HERE
    outs = []
    for salt in ("1", "2"):
        env = dict(os.environ, PYTHONHASHSEED=salt)
        outs.append(subprocess.run([sys.executable, "-c", code], env=env, check=True, capture_output=True,
                                   text=True).stdout.strip())
    assert outs[0] == outs[1] and len(outs[0].split(",")) == 10
