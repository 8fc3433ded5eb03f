"""The column-parallel oracle driver (used for the stored values of the large
workloads) equals the serial oracle up to the reassociation of the final sum over
column ranges, for plain and Jacobi-preconditioned CG."""
import numpy as np
import pytest

import gen
from oracle import erc as OE
from oracle.parallel import resistance_parallel


@pytest.mark.parametrize("precond", ["none", "jacobi"])
def test_parallel_equals_serial(precond):
    g = gen.erdos_renyi(400, 0.02, 5, weighted=True)
    args = (g, 48, 16, 1e-5, 1e-8, 2000, 9, "f64")
    R_ser, info = OE.resistance(*args, precond=precond)
    R_par, iters, conv = resistance_parallel(*args, col_begin=0, col_end=48, procs=3,
                                             precond=precond)
    assert conv.all()
    np.testing.assert_array_equal(iters, np.concatenate(info.iters))
    assert np.max(np.abs(R_par - R_ser) / R_ser) < 1e-14
