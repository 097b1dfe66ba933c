"""Helpers shared by the GPU tests: run the library through its C ABI on
numpy inputs and compare with the oracle to the stated bar."""
import numpy as np
import torch

import oracle
import paper_2212_00404_amd as dc

# fp32 results must satisfy |O - O64| <= REL * sum|I*F| for every output.
REL = 1e-5


def dev():
    return torch.device("cuda:0")


def gpu_single(I, F, **kw):
    It = torch.from_numpy(np.ascontiguousarray(I)).to(dev())
    Ft = torch.from_numpy(np.ascontiguousarray(F)).to(dev())
    O = dc.single(It, Ft, **kw)
    torch.cuda.synchronize()
    return O.cpu().numpy()


def gpu_multi(I, F, variant="auto", **kw):
    It = torch.from_numpy(np.ascontiguousarray(I)).to(dev())
    Ft = torch.from_numpy(np.ascontiguousarray(F)).to(dev())
    O = dc.multi(It, Ft, variant=variant, **kw)
    torch.cuda.synchronize()
    return O.cpu().numpy()


def assert_within(O, O64, A64, what, rel=REL):
    assert O.shape == O64.shape, "%s: shape %r vs %r" % (what, O.shape, O64.shape)
    assert np.isfinite(O).all(), "%s: non-finite output" % what
    err = np.abs(O.astype(np.float64) - O64)
    bound = rel * A64
    bad = err > bound
    if bad.any():
        idx = np.unravel_index(np.argmax(err - bound), O.shape)
        raise AssertionError("%s: %d of %d outputs outside %g*sum|I*F|; worst at %r: gpu %r "
                             "oracle %r bound %r" % (what, bad.sum(), O.size, rel, idx, O[idx],
                                                     O64[idx], bound[idx]))


def assert_exact(O, O64, what):
    """Bit-exact by value (+0 and -0 compare equal)."""
    assert O.shape == O64.shape, "%s: shape %r vs %r" % (what, O.shape, O64.shape)
    diff = O.astype(np.float64) != O64
    if diff.any():
        idx = np.unravel_index(np.argmax(diff), O.shape)
        raise AssertionError("%s: %d mismatches; first at %r: gpu %r oracle %r"
                             % (what, diff.sum(), idx, O[idx], O64[idx]))


def oracle_single(I, F):
    return oracle.conv_single(I, F)


def oracle_multi(I, F):
    return oracle.conv_multi(I, F)
