"""Host-side behaviour of the binding's cached workspaces (no GPU): a
workspace that a larger call replaces stays referenced, so a HIP graph
captured with it can never write into memory handed to another tensor."""
import gc
import weakref

import torch

from paper_2606_18394_amd import binding


def test_superseded_workspace_stays_referenced():
    key = ("test-host", "cpu", 12345)
    binding._workspaces.pop(key, None)
    first = binding.workspace("test-host", 1000, "cpu", 12345)
    assert first.numel() >= 1000 and int(first.sum()) == 0
    ptr = first.data_ptr()
    ref = weakref.ref(first)
    del first
    gc.collect()
    same = binding.workspace("test-host", 800, "cpu", 12345)     # fits: no growth
    assert same.data_ptr() == ptr
    del same
    grown = binding.workspace("test-host", 5000, "cpu", 12345)   # grows: a new buffer
    assert grown.numel() >= 5000 and grown.data_ptr() != ptr
    gc.collect()
    old = ref()
    assert old is not None, "the superseded workspace was freed"
    assert old.data_ptr() == ptr
    assert any(t is old for t in binding._retired)
    binding._workspaces.pop(key, None)


def test_workspaces_are_per_stream():
    a = binding.workspace("test-host2", 300, "cpu", 1)
    b = binding.workspace("test-host2", 300, "cpu", 2)
    assert a.data_ptr() != b.data_ptr()
    for k in [("test-host2", "cpu", 1), ("test-host2", "cpu", 2)]:
        binding._workspaces.pop(k, None)
