"""Host-staged transfer (the paper's sender / receiver staging options, Sec.
3.3): the packing kernel writes its per-receiver regions into pinned host
memory and the assembly kernel reads them from there over PCIe. Results must
be bit-identical to the device-resident path and to the oracle."""

import numpy as np
import pytest

import synthetic_checkpoint as sc
import paper_2609_25442_amd as wb
from oracle.layout import layout_from_spec
from synthetic_checkpoint.workloads import scaled

from gpu_util import roundtrip

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", ["send", "recv", "both"])
@pytest.mark.parametrize("name", ["llama3_8b_fsdp8_to_tp1", "llama3_8b_tp4_to_tp2", "mixtral_ep8fsdp2_to_ep2",
                                  "dsv3_ep64_to_ep8_fp8"])
def test_host_staged_parity(name, mode):
    """Sender staging only, receiver staging only, or both (the fourth mode,
    neither, is the device-resident parity test)."""
    w = scaled(name)
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    cat = otr.catalog
    dt = w["trainer"]["dtype"]
    cache = {}

    def values(t):
        if t not in cache:
            cache[t] = sc.values_numpy(t, np.arange(cat[t].numel), dt).reshape(cat[t].rows, cat[t].cols)
        return cache[t]

    roundtrip(otr, oro, values, wb.Layout.describe(w["model"], w["trainer"]),
              wb.Layout.describe(w["model"], w["rollout"]), label=f"staged-{mode}-{name}",
              staged=True if mode == "both" else mode)
