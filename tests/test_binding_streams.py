"""The binding allocates a call's workspace and new outputs on the stream the
call runs on (so torch's caching allocator does not hand them to other work
while the call's kernels still use them).  Checked on the CPU with a stand-in
for torch.cuda: allocations are recorded with the stream that was current."""

import contextlib

import paper_2609_00355_amd as G


class _FakeCuda:
    def __init__(self):
        self.current = "default"
        self.log = []

    def current_stream(self, device=None):
        return self.current

    @contextlib.contextmanager
    def stream(self, s):
        prev, self.current = self.current, s
        try:
            yield
        finally:
            self.current = prev


class _FakeTorch:
    uint8 = "uint8"

    def __init__(self):
        self.cuda = _FakeCuda()

    def empty(self, shape, dtype=None, device=None):
        self.cuda.log.append(("empty", shape, self.cuda.current))
        return ("tensor", shape)


def test_workspace_and_outputs_follow_the_call_stream(monkeypatch):
    fake = _FakeTorch()
    monkeypatch.setattr(G, "_torch", lambda: fake)
    G._workspace(1000, "cuda:0", None, stream="side")
    G._new_output(fake.empty, (4, 4), "side", dtype="f32", device="cuda:0")
    G._workspace(1000, "cuda:0", None)             # no stream: the current one
    G._new_output(fake.empty, (2,), None, dtype="f32", device="cuda:0")
    G._workspace(1000, "cuda:0", None, stream="default")  # the current stream itself
    assert [entry[2] for entry in fake.cuda.log] == ["side", "side", "default", "default", "default"]
    assert fake.cuda.current == "default"
    # a caller's workspace is used as given
    ws = ("tensor", "mine")
    assert G._workspace(10, "cuda:0", ws, stream="side") is ws
