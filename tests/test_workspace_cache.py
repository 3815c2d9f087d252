"""Host logic of the binding's cached workspace (no GPU: the stream lookup and the
size query are stubbed, buffers live on the CPU).  One buffer per (device,
stream), reused while large enough; a larger request replaces it and the old
buffer stays referenced, so a HIP graph captured with its address can still be
replayed after a larger layer call."""
import os
import sys
import types

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

from paper_2609_05228_amd import layer  # noqa: E402


def test_workspace_cache_keeps_superseded_buffers(monkeypatch):
    sizes = {}
    monkeypatch.setattr(layer._lib, "workspace_size", lambda desc: sizes["n"])
    streams = {"cur": 11}
    monkeypatch.setattr(layer.torch.cuda, "current_stream",
                        lambda dev=None: types.SimpleNamespace(cuda_stream=streams["cur"]))
    monkeypatch.setattr(layer, "_WS_CACHE", {})
    monkeypatch.setattr(layer, "_WS_RETIRED", [])
    dev = torch.device("cpu")
    sizes["n"] = 1000
    a = layer.workspace(None, dev)
    assert a.numel() == 1000 and a.dtype == torch.uint8
    sizes["n"] = 600
    assert layer.workspace(None, dev) is a            # large enough: reused
    sizes["n"] = 5000
    b = layer.workspace(None, dev)
    assert b is not a and b.numel() == 5000
    assert any(r is a for r in layer._WS_RETIRED)     # the old buffer stays allocated
    sizes["n"] = 10
    assert layer.workspace(None, dev).numel() == 5000  # never shrinks; at least 256 bytes
    streams["cur"] = 12                                # another stream: its own buffer
    c = layer.workspace(None, dev)
    assert c is not b and c.numel() == 256
