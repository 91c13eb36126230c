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


@pytest.mark.parametrize("policy,n", [("marginal", 4), ("exhaustive", 2), ("joint", 5), ("joint", 8)])
def test_cost_table_too_short(policy, n):
    """The per-sequence rules read cost[0..G] and the joint rule cost[0..B*G]: shorter tables are
    refused (B = 2, G = 4 here)."""
    with pytest.raises(ValueError, match="cost entries"):
        decode.DecodeLoop(None, None, None, 128, 2, 4, policy, None, cost=[1.0] * n)


def test_binding_checks_selector_tables():
    """lsv.py refuses selector tables that are not contiguous cuda tensors of the right dtype and
    length before the call reaches the library (a short table would be read past its end on the
    device).  Without a GPU only the host-tensor refusal can be shown here."""
    import torch

    from paper_2608_08721_amd import lsv
    conf = torch.zeros((2, 4), dtype=torch.float32)
    for cost in (torch.ones(4, dtype=torch.float64), torch.ones(5, dtype=torch.float32),
                 torch.ones(5, dtype=torch.float64)):  # host tensors are refused too
        with pytest.raises(lsv.LsvError, match="cost|conf"):
            lsv.lsv_select_length(lsv.LSV_SEL_MARGINAL, 2, 4, conf, cost, 1, 4, 2.0, 4, 0, 0, None, None, None,
                                  stream=0)
    with pytest.raises(lsv.LsvError, match="cost|conf"):
        lsv.lsv_select_joint(2, 4, conf, torch.ones(8, dtype=torch.float64), 4, 0, 0, None, None, None, stream=0)
