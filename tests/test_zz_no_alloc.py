"""fc_retrieve_noalloc (the retrieval for callers that cannot allocate: its
workspace is the library's static per-GPU array) gives exactly what
fc_retrieve gives with a caller workspace, on two calls in a row, the second
with a smaller batch (the static array keeps the first call's contents)."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_17139_amd as fc  # noqa: E402

P = dict(synth.PARAMS)


def _outputs(B, S, k, m, fill):
    out = fc.retrieve_outputs(B, S, k, m, torch.device("cuda"))
    for v in out.values():
        v.view(torch.uint8).fill_(fill)
    return out


def test_noalloc_matches_retrieve():
    print("noalloc: stores", flush=True)
    tp, tg = synth.store(2, "project"), synth.store(1, "single")
    stores = [fc.Store(torch.from_numpy(tp).cuda(), pair_vocab=synth.VOCAB, records=True),
              fc.Store(torch.from_numpy(tg).cuda(), pair_vocab=synth.VOCAB)]
    ctx_all = torch.from_numpy(synth.queries(2)).cuda()
    kw = dict(n_max=P["n_max"], n_min=P["n_min"], k=P["k"], m=P["m"])
    for B, lo in ((256, 0), (37, 200)):
        print(f"noalloc: B={B}", flush=True)
        ctx = ctx_all[lo:lo + B].contiguous()
        want = fc.fc_retrieve(stores, ctx, out=_outputs(B, 2, P["k"], P["m"], 0xAB), **kw)
        got = fc.fc_retrieve_noalloc(stores, ctx, out=_outputs(B, 2, P["k"], P["m"], 0xAB), **kw)
        torch.cuda.synchronize()
        assert int(want["taken"].sum()) > 0
        for f in fc.RETRIEVE_FIELDS:
            assert torch.equal(got[f], want[f]), (B, f)
