"""Pins the oracle's Philox4x32-10 to an independent implementation: the
host-callable Philox engine of AMD's rocRAND library (its ten-round block
function, read through a subclass), compiled here for the host CPU.  The
oracle's round function must give the same four words for every counter and
key, including the all-zero and all-ones corner cases (Salmon et al., SC'11,
the generator the sampler's noise is defined by)."""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

from oracle.philox import philox4x32_10

_SRC = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
struct Block : rocrand_device::philox4x32_10_engine {
  uint4 run(uint4 c, uint2 k) { return ten_rounds(c, k); }
};
int main() {
  unsigned c0, c1, c2, c3, k0, k1;
  Block b;
  while (std::scanf("%u %u %u %u %u %u", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
    uint4 c; c.x = c0; c.y = c1; c.z = c2; c.w = c3;
    uint2 k; k.x = k0; k.y = k1;
    const uint4 r = b.run(c, k);
    std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
"""


def _hipcc():
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


def test_philox_equals_rocrand_block_function():
    hipcc = _hipcc()
    if hipcc is None or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("rocRAND headers / hipcc not available")
    rng = np.random.default_rng(11)
    ctr = rng.integers(0, 2 ** 32, size=(3000, 4), dtype=np.uint64)
    key = rng.integers(0, 2 ** 32, size=(3000, 2), dtype=np.uint64)
    ctr[0], key[0] = 0, 0
    ctr[1], key[1] = 0xFFFFFFFF, 0xFFFFFFFF
    ctr[2] = [5, 17, 0, 0]                 # the sampler's form: (v >> 2, position, uid lo, uid hi)
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "philox_ref.cpp")
        exe = os.path.join(d, "philox_ref")
        open(src, "w").write(_SRC)
        subprocess.check_call([hipcc, "-x", "hip", "--offload-arch=gfx950", "-O1", src, "-o", exe],
                              stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
        inp = "\n".join(" ".join(str(int(v)) for v in (*ctr[i], *key[i])) for i in range(len(ctr)))
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
    ref = np.array([[int(t) for t in line.split()] for line in out.strip().splitlines()], np.uint64)
    got = np.stack(philox4x32_10(ctr[:, 0], ctr[:, 1], ctr[:, 2], ctr[:, 3], key[:, 0], key[:, 1]),
                   axis=1).astype(np.uint64)
    np.testing.assert_array_equal(got, ref)
