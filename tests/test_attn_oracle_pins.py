"""The attention oracle against its pins (no GPU)."""
import pytest

import oracle
from tests import attn_pins


@pytest.mark.parametrize("name", sorted(attn_pins.ALL_CHECKS))
def test_attention_oracle_pin(name):
    fails = attn_pins.ALL_CHECKS[name](oracle.lib())
    assert not fails, fails[:5]
