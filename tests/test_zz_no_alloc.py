"""eb_decode_step_noalloc, the decode step for callers that cannot allocate device memory,
against eb_decode_step with a caller workspace: every output bit for bit, on two calls in a row
on one device, the second with a smaller step (the library's scratch keeps the first call's
contents, which must not matter)."""
import sys

import numpy as np
import pytest
import torch

from paper_2609_16450_amd import (EB_NOALLOC_SCRATCH_BYTES, eb_decode_step,
                                  eb_decode_step_noalloc, eb_decode_step_workspace)
from paper_2609_16450_amd.device_case import DeviceStep
from workloads import make_step

pytestmark = pytest.mark.gpu

OUTPUTS = ("attn_out", "conf", "entropy", "argmax", "max_logit", "unmask", "tokens", "masked",
           "n_commit", "resolved")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_noalloc_step_equals_step_two_calls_second_smaller():
    # first a batch-16 step (tile LM head, fused epilogue), then the batch-1 step (streaming LM
    # head with the attention inside its launch, key-split partials in the scratch)
    for name in ("llada8b_b16", "llada8b_b1"):
        say(f"noalloc step workload={name}")
        case = make_step(name)
        ref = DeviceStep(case)
        got = DeviceStep(case)
        need = eb_decode_step_workspace(ref.buffers)
        assert 0 < need <= EB_NOALLOC_SCRATCH_BYTES
        eb_decode_step(ref.buffers)
        eb_decode_step_noalloc(got.buffers)
        torch.cuda.synchronize()
        for k in OUTPUTS:
            a, b = getattr(ref, k), getattr(got, k)
            assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.uint8) if b.dtype == torch.bfloat16 else b), (name, k)
        # the step did work: some rows committed
        assert int(got.unmask.sum()) > 0
        assert np.array_equal(ref.tokens.cpu().numpy(), got.tokens.cpu().numpy())
