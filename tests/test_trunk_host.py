"""Host-side argument checks of the trunk orchestrator (no GPU call is made: the
constructor rejects these before it allocates anything)."""
import pytest

from paper_2607_02829_amd import inputs
from paper_2607_02829_amd.trunk import Trunk

pytestmark = pytest.mark.cpu


def test_trunk_rejects_bad_arguments():
    w = inputs.small("trunk_s")
    params = inputs.params_to_storage(inputs.block_params(w, 3), w.dtype)
    with pytest.raises(ValueError):
        Trunk(w, (0, 2, 1), params)                        # an empty stage
    with pytest.raises(ValueError):
        Trunk(w, (1, 1, 1), params[:2])                    # parameters for 2 of 3 blocks
    with pytest.raises(ValueError):
        Trunk(w, (1, 1, 1), params, K=w.L + 1)             # K beyond L
    with pytest.raises(ValueError):
        Trunk(w.with_(kind="adaln"), (1, 1, 1), params)    # pre-LN blocks only
    with pytest.raises(ValueError):
        Trunk(w, (1, 1, 1), params, select="gradient")     # random or attention-score selection
    with pytest.raises(ValueError):
        Trunk(w, (1, 1, 1), params, checkpoint="yes")      # checkpointing is on or off
