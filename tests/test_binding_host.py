"""Host-side checks of the Python binding that run before any library call."""

import types

import pytest
import torch

from paper_2608_15533_amd import deltalog as D


@pytest.mark.parametrize("entry", ["eager", "append", "merge", "tiled"])
def test_token_with_fewer_rows_than_the_slot_list_is_refused(entry):
    """Token row i drives slots[i]: a token of 2 rows with a list of 4 slots would make the
    kernel read past the token's arrays, so the binding raises before calling the library
    (the slot list here is a host tensor: the row check comes first)."""
    desc = D.make_desc("gdn", 8, 2, 128, 128, 16, "bf16")
    tok = types.SimpleNamespace(n=2)
    slots = torch.arange(4, dtype=torch.int32)
    with pytest.raises(ValueError, match="token holds 2 rows but the launch drives 4"):
        if entry == "eager":
            D.dl_eager_step(desc, None, tok, None, slots=slots)
        elif entry == "append":
            D.dl_append_step(desc, None, tok, None, slots=slots)
        elif entry == "merge":
            D.dl_merge(desc, None, tok, None, slots=slots)
        else:
            D.dl_append_step_tiled(desc, None, tok, None, slots=slots)


def test_token_rows_without_a_slot_list():
    """Without a slot list the launch drives the token's rows; more token rows than the
    slot list holds are allowed (the extra rows are not read)."""
    desc = D.make_desc("gdn", 8, 2, 128, 128, 16, "bf16")
    assert D._rows(desc, None, 8) == (None, 8)
    assert D._rows(desc, None, None) == (None, 8)
    with pytest.raises(ValueError, match="must be a device tensor"):
        D._rows(desc, torch.arange(3, dtype=torch.int32), 8)   # passes the row check
