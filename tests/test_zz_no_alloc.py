"""gnn_softmax_xent_noalloc (the variant of gnn_softmax_xent for callers that
cannot allocate) against gnn_softmax_xent on the same inputs, through the C
ABI: two calls in a row, the second with fewer rows, so that the library's
scratch array holds the first call's contents when the second runs."""
import numpy as np
import pytest
import torch

from tests import gpu_common as gc

pytestmark = pytest.mark.gpu


def test_softmax_xent_noalloc_matches_workspace_entry_point():
    from paper_2403_17092_amd import gnnhip
    dev = gc.device()
    g = torch.Generator().manual_seed(7)
    for B, C in ((3000, 47), (700, 172)):
        gc.announce("softmax xent noalloc", B, C)
        logits = (torch.randn(B, C, generator=g) * 3).to(dev)
        labels = torch.randint(0, C, (B,), generator=g, dtype=torch.int32).to(dev)
        loss_ref, dl_ref = gnnhip.softmax_xent(logits, labels)
        dl = torch.full_like(logits, float("nan"))
        loss = torch.full((1,), float("nan"), device=dev)
        gnnhip.softmax_xent_noalloc(logits, labels, dl, loss)
        torch.cuda.synchronize()
        assert gnnhip.check_errors() == 0
        # the same kernels in the same order: identical results
        np.testing.assert_array_equal(dl.cpu().numpy(), dl_ref.cpu().numpy())
        assert loss.item() == loss_ref.item()
        # and both are the mean softmax cross-entropy (float64 on the host)
        z = logits.double().cpu().numpy()
        y = labels.long().cpu().numpy()
        m = z.max(axis=1, keepdims=True)
        lse = m[:, 0] + np.log(np.exp(z - m).sum(axis=1))
        want = float(np.mean(lse - z[np.arange(B), y]))
        assert abs(loss.item() - want) <= 1e-5 * abs(want)


def test_softmax_xent_noalloc_rejects_too_many_rows():
    from paper_2403_17092_amd import gnnhip
    dev = gc.device()
    B = 65537
    logits = torch.zeros(B, 4, device=dev)
    labels = torch.zeros(B, dtype=torch.int32, device=dev)
    with pytest.raises(gnnhip.GnnError):
        gnnhip.softmax_xent_noalloc(logits, labels, torch.empty_like(logits),
                                    torch.zeros(1, device=dev))
