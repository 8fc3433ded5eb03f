"""The C ABI used from plain C (tests/c_abi/erc_example.c): buffers sized by the *_bytes
queries and allocated with hipMalloc, then erc_create, erc_resistance, erc_curvature,
erc_sampling_probs and erc_edge_endpoints on a random weighted tree, checked inside the
C code against closed forms that hold for every projection on a tree (Section 3.1.2: a
bridge's sketched resistance is 1/w; then Eq. 2 and Eqs. 7-8).  The C code is a shared
library built by __graft_entry__.build(), called here through ctypes."""
import ctypes
import os

import pytest

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "liberc_example.so")


@pytest.mark.parametrize("n,seed", [(2000, 5), (2, 1)])
def test_c_program_on_a_tree(n, seed):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(LIB), f"{LIB} missing: run __graft_entry__.build()"
    lib = ctypes.CDLL(LIB)
    fn = lib.erc_example_tree
    fn.argtypes = [ctypes.c_int32, ctypes.c_uint64, ctypes.c_char_p, ctypes.c_int32]
    fn.restype = ctypes.c_int
    buf = ctypes.create_string_buffer(512)
    rc = fn(n, seed, buf, len(buf))
    msg = buf.value.decode()
    print(msg)
    assert rc == 0, msg
