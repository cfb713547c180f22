"""Host-only checks of the C ABI: the library loads, exports every function
declared in include/entwine.h, validates arguments, and its exported
traversal / consumer maps equal the oracle's (Equation 1 and the comparison
orders).  No GPU call is made."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import schedule as S
from paper_2609_11562_amd import entwine as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(E.lib_path()):
        from paper_2609_11562_amd import build
        build.build()
    return E.lib()


def _declared_functions():
    with open(os.path.join(ROOT, "include", "entwine.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(entwine_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(E._PROTOS), "binding and header disagree"


def test_abi_version_and_strings(lib):
    assert lib.entwine_abi_version() == 3
    assert ctypes.sizeof(E.Config) == 12 * 4
    assert E._status_name(E.ETIMEOUT) == "ENTWINE_ETIMEOUT"
    c = E.Config.make()
    assert (c.order, c.gemm_cfg, c.withhold_peer) == (E.ORDER_INTERLEAVED, -1, -1)


@pytest.mark.parametrize("M,N,K,P,dest,want", [
    (512, 1024, 256, 2, 0, E.OK),
    (512, 1024, 256, 2, -1, E.OK),
    (4096, 4096, 1376, 8, 7, E.OK),
    (512, 1024, 256, 2, 2, E.EINVAL),          # dest out of range
    (512, 1024, 256, 2, -2, E.EINVAL),
    (384, 1024, 256, 2, 0, E.EINVAL),          # M not a multiple of 128 P
    (512, 1000, 256, 2, 0, E.EINVAL),          # N not a multiple of 128
    (512, 1024, 250, 2, 0, E.EINVAL),          # K not a multiple of 8
    (512, 1024, 0, 2, 0, E.EINVAL),
    (1152, 1024, 64, 9, 0, E.EINVAL),          # P above the maximum
    (512, 1024, 64, 0, 0, E.EINVAL),
])
def test_validate_shapes(lib, M, N, K, P, dest, want):
    assert E.validate(M, N, K, P, dest) == want


def test_validate_config(lib):
    ok = E.validate(512, 1024, 256, 2, 0, E.Config.make(gemm_cfg=E.GEMM_128x128))
    assert ok == E.OK
    # 256-row blocks do not divide a 128-row chunk.
    assert E.validate(256, 1024, 64, 2, 0, E.Config.make(gemm_cfg=E.GEMM_256x256)) == E.EUNSUPPORTED
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(order=3)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(reduce_threads=64)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(withhold_peer=1)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(withhold_peer=0)) == E.OK
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(launch=3)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(launch=2)) == E.OK
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(reduce_wgs=-1)) == E.OK
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(reduce_wgs=-1, launch=1)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(reduce_wgs=-2)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(release_blocks=-1, store_mode=1)) == E.OK
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(release_blocks=E.RELEASE_PARTITION)) == E.OK
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(release_blocks=E.RELEASE_OUTPUT)) == E.OK
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(release_blocks=-4)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(store_mode=2)) == E.OK
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(store_mode=3)) == E.EINVAL
    assert E.validate(512, 1024, 256, 2, 0, E.Config.make(launch=1)) == E.OK


SHAPES = [(512, 1024, 2, 256, 256), (4096, 4096, 8, 256, 256), (4096, 4096, 8, 128, 128),
          (8192, 8192, 8, 256, 128), (1024, 768, 4, 128, 256), (512, 768, 4, 128, 256),
          (1536, 512, 3, 256, 128), (16384, 8192, 8, 256, 256)]


@pytest.mark.parametrize("M,N,P,BM,BN", SHAPES)
@pytest.mark.parametrize("order", [S.INTERLEAVED, S.ROW_MAJOR, S.M_MAJOR])
@pytest.mark.parametrize("group_m", [1, 2, 4, 8])
def test_library_schedule_matches_oracle(lib, M, N, P, BM, BN, order, group_m):
    blocks, tiles = E.tile_schedule(order, M, N, P, BM, BN, group_m)
    ref = S.full_schedule(order, M, N, P, BM, BN, group_m)
    assert blocks.tolist() == [[d, l, mb, nb] for d, l, mb, nb, _ in ref]
    want = np.full(tiles.shape, -1, np.int32)
    for d, _, _, _, tl in ref:
        for t, tr, tc in tl:
            want[tr, tc] = (d, t)
    assert np.array_equal(tiles, want)


@pytest.mark.parametrize("P,Q,x", [(4, 6, 2), (8, 128, 16), (2, 16, 3), (8, 512, 32), (1, 9, 4)])
def test_library_consumer_tasks_match_oracle(lib, P, Q, x):
    for j in range(x):
        assert E.consumer_tasks(P - 1, P, Q, x, j) == (P - 1, S.consumer_tasks(j, x, Q))
    xa = x * P
    for j in range(xa):
        d, tasks = S.all_chunk_consumer_tasks(j, xa, P, Q)
        assert E.consumer_tasks(E.DEST_ALL, P, Q, xa, j) == (d, tasks)


def test_schedule_rejects_bad_blocks(lib):
    with pytest.raises(E.EntwineError):
        E.tile_schedule(0, 512, 1024, 2, 512, 256)
    with pytest.raises(E.EntwineError):
        E.tile_schedule(0, 512, 1024, 2, 256, 256, 65)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(E, "_LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(E, "_lib", None)
    with pytest.raises(ImportError):
        E.lib()


def test_header_is_plain_c(tmp_path):
    """The ABI header compiles as C (no C++ types leak into the boundary)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use.c"
    src.write_text('#include "entwine.h"\n'
                   'int main(void) { entwine_config c; entwine_config_default(&c);\n'
                   '  return entwine_abi_version() == ENTWINE_ABI_VERSION && c.launch == 0 ? 0 : 1; }\n')
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-I", inc, str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
