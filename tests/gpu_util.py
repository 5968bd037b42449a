"""Helpers shared by the GPU parity tests: mirror oracle caches onto the
device, compare results element by element, and print what a case is before
it runs (so a failing GPU step names itself)."""
import sys

import numpy as np
import torch

from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

ERR_OF_STATUS = {0: 0, 1: sm.ERR_EINVAL, 2: sm.ERR_ERANGE, 3: sm.ERR_ENOMEM}
TOL = {torch.float32: 1e-5, torch.bfloat16: 1e-2}


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def dev():
    return torch.device("cuda:0")


def rel_l2_max(got, ref):
    """max over vectors (last axis) of ||got - ref|| / ||ref||; a zero
    reference vector requires an exactly zero result."""
    got = np.asarray(got, np.float64).reshape(-1, np.shape(ref)[-1])
    ref = np.asarray(ref, np.float64).reshape(-1, np.shape(ref)[-1])
    num = np.linalg.norm(got - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    zero = den == 0
    if np.any(zero) and np.any(num[zero] != 0):
        return np.inf
    den[zero] = 1.0
    return float(np.max(num / den)) if len(num) else 0.0


def raw_to_torch(a, device):
    return wl.from_raw(a, device)


def gpu_cache_like(oc, dtype):
    """GPU PagedCache whose whole state is a copy of oracle cache ``oc``."""
    c = sm.PagedCache(dtype=dtype, num_kv_heads=oc.H, head_dim=oc.D, block_size=oc.bs,
                      num_blocks=oc.num_blocks, max_seqs=oc.max_seqs,
                      max_blocks_per_seq=oc.max_blocks, device=dev())
    sync_gpu_from_oracle(c, oc)
    return c


def sync_gpu_from_oracle(c, oc):
    c.k_pool.copy_(raw_to_torch(oc.k_pool, dev()))
    c.v_pool.copy_(raw_to_torch(oc.v_pool, dev()))
    c.block_table.copy_(torch.from_numpy(oc.block_table))
    c.lengths.copy_(torch.from_numpy(oc.lengths))
    c.free_stack.copy_(torch.from_numpy(oc.free_stack))
    c.free_top.copy_(torch.from_numpy(oc.free_top))
    c.err.zero_()
    torch.cuda.synchronize()


def assert_same_state(c, oc, pools=True):
    torch.cuda.synchronize()
    np.testing.assert_array_equal(c.lengths.cpu().numpy(), oc.lengths)
    np.testing.assert_array_equal(c.block_table.cpu().numpy(), oc.block_table)
    top = int(oc.free_top[0])
    assert int(c.free_top.item()) == top
    np.testing.assert_array_equal(c.free_stack.cpu().numpy()[:top], oc.free_stack[:top])
    if pools:
        assert np.array_equal(wl.to_raw(c.k_pool), oc.k_pool), "K pool differs"
        assert np.array_equal(wl.to_raw(c.v_pool), oc.v_pool), "V pool differs"


def i32(a):
    return torch.as_tensor(np.asarray(a, np.int32)).to(dev())
