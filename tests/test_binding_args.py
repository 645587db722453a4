"""Decoder.decode's argument checks (CPU): arguments the C call would misread
-- another integer width, rank, row count or device -- raise DcError before
anything is launched."""
import numpy as np
import pytest
import torch

import paper_2609_35115_amd as dc

B, MAXN, FPT = 3, 25, 2


def check(tokens, f0=None, host=False, source=False, device=0):
    return dc.check_decode_args(tokens, f0, B, MAXN, FPT, source, host, device)


def status_of(fn):
    with pytest.raises(dc.DcError) as e:
        fn()
    return e.value.status


def test_good_arguments_give_n():
    ids = np.zeros((B, 7), dtype=np.int32)
    assert check(ids, host=True) == 7
    assert check(ids) == 7                                # numpy is copied to the device
    assert check(ids.astype(np.int64)) == 7               # ... from any integer type whose values fit
    assert check(ids, np.zeros((B, 14), np.float32), host=True, source=True) == 7
    assert check(ids[:, ::2]) == 4                        # a strided view is copied as well


def test_shape_and_count():
    assert status_of(lambda: check(np.zeros((B + 1, 4), np.int32))) == dc.DC_EINVAL   # short/long batch
    assert status_of(lambda: check(np.zeros((B - 1, 4), np.int32))) == dc.DC_EINVAL
    assert status_of(lambda: check(np.zeros((B * 4,), np.int32))) == dc.DC_EINVAL      # rank 1
    assert status_of(lambda: check(np.zeros((B, 0), np.int32))) == dc.DC_EINVAL        # n = 0
    assert status_of(lambda: check(np.zeros((B, MAXN + 1), np.int32))) == dc.DC_ERANGE  # n > max_tokens
    assert status_of(lambda: check(None)) == dc.DC_EINVAL


def test_integer_width_and_kind():
    # host mode reads the array in place: only int32 is accepted
    assert status_of(lambda: check(np.zeros((B, 4), np.int64), host=True)) == dc.DC_EINVAL
    assert status_of(lambda: check(np.zeros((B, 4), np.float32))) == dc.DC_EINVAL
    big = np.zeros((B, 4), np.int64)
    big[1, 2] = 2 ** 31
    assert status_of(lambda: check(big)) == dc.DC_EINVAL
    # torch tensors are passed by address: int64 (torch's default) would be read as int32 pairs
    assert status_of(lambda: check(torch.zeros((B, 4), dtype=torch.int64))) == dc.DC_EINVAL


def test_device_of_tensors():
    # a host tensor in device mode would be dereferenced as a device address
    assert status_of(lambda: check(torch.zeros((B, 4), dtype=torch.int32))) == dc.DC_EINVAL
    # a tensor in host mode likewise
    assert status_of(lambda: check(torch.zeros((B, 4), dtype=torch.int32), host=True)) == dc.DC_EINVAL


def test_f0_of_a_source_decoder():
    ids = np.zeros((B, 5), np.int32)
    assert status_of(lambda: check(ids, None, source=True)) == dc.DC_EINVAL
    assert status_of(lambda: check(ids, np.zeros((B, 5), np.float32), source=True)) == dc.DC_EINVAL   # n, not n*fpt
    assert status_of(lambda: check(ids, np.zeros((B, 10), np.float64), host=True, source=True)) == dc.DC_EINVAL
    assert status_of(lambda: check(ids, np.zeros((B, 10), np.int32), source=True)) == dc.DC_EINVAL
    assert status_of(lambda: check(ids, torch.zeros((B, 10)), source=True)) == dc.DC_EINVAL         # host tensor
    assert status_of(lambda: check(ids, np.zeros((B, 10), np.float32))) == dc.DC_EINVAL              # no source
