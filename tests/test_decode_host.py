"""Host-side checks of the decoding loop driver (no GPU): bad policies and missing cost
tables are refused before any device buffer is made."""
import pytest

from paper_2608_08721_amd import decode


def test_rejects_unknown_policy():
    with pytest.raises(ValueError, match="policy"):
        decode.DecodeLoop(None, None, None, 128, 1, 4, "fastest", None)


@pytest.mark.parametrize("policy", ["marginal", "exhaustive"])
def test_cost_table_required(policy):
    with pytest.raises(ValueError, match="cost"):
        decode.DecodeLoop(None, None, None, 128, 1, 4, policy, None)
