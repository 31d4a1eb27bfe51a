"""The anchor-path parity tests can fail: on each anchor-dominant workload
the GPU tests use, gathering every anchor row for the wrong token (ids
permuted), or decoding with the sender's table instead of the receiver's,
moves the oracle's outputs by at least five times the bf16 tolerance
(Eqs. 1-2; the anchor is E_small[ids] P with P frozen orthonormal, Eq. 3).
CPU only: oracle and generator."""
import pytest

from _helpers import ANCHOR_CASES, BF16_TOL, anchor_case, anchor_discrimination, oracle_payload


@pytest.mark.parametrize("name", sorted(ANCHOR_CASES))
def test_wrong_anchor_rows_exceed_gate(name):
    x, rx, C = anchor_case(name)
    disc = anchor_discrimination(x, oracle_payload(x, C), C, rx)
    print(name, {k: round(v, 3) for k, v in disc.items()})
    for key, v in disc.items():
        assert v >= 5 * BF16_TOL, (key, v)
