"""SSD tier: the native asynchronous chunk store and the queue-window prefetch harness
(Sec. 4.4), on the CPU. Files live in a scratch folder inside the repository."""
import os
import shutil
import tempfile

import numpy as np
import pytest

from paper_2603_23049_amd import pcr, prefetch, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture
def scratch():
    base = os.path.join(ROOT, ".pytest_store")
    os.makedirs(base, exist_ok=True)
    d = tempfile.mkdtemp(dir=base)
    yield d
    shutil.rmtree(d, ignore_errors=True)


def test_store_round_trip_async(scratch):
    cb = 64 * 1024
    st = pcr.ChunkStore(os.path.join(scratch, "kv.bin"), cb, io_threads=3)
    src = [prefetch.chunk_pattern(i, cb) for i in range(6)]              # numpy: not page-aligned
    aligned = prefetch.page_aligned_buffer(cb)
    aligned[:] = prefetch.chunk_pattern(99, cb)
    for i, buf in enumerate(src):
        st.write_async(10 + 3 * i, buf)
    st.write_async(7, aligned)
    dst = [prefetch.page_aligned_buffer(cb) for _ in range(7)]
    for i in range(6):
        st.read_async(10 + 3 * i, dst[i])        # waits for its own write first
    st.read_async(7, dst[6])
    st.wait()
    for i in range(6):
        assert np.array_equal(dst[i], src[i])
    assert np.array_equal(dst[6], aligned)
    s = st.stats()
    assert s["bytes_written"] == 7 * cb and s["bytes_read"] == 7 * cb
    with pytest.raises(pcr.PcrError):
        st.read_async(1000, dst[0])              # never written
    with pytest.raises(ValueError):
        st.write_async(1, np.zeros(cb - 1, np.uint8))
    st.close()


def test_window_prefetch_serves_correct_bytes_and_cuts_on_demand_reads(scratch):
    stream = synth.rag_stream(4, n_requests=64 + 30)
    kw = dict(chunk_bytes=16 * 1024, dram_chunks=48, compute_ms_per_token=0.0005, warm=64, io_threads=4,
              verify=True)
    s0 = prefetch.serve(stream.requests, store_path=os.path.join(scratch, "w0.bin"), window=0, **kw)
    s4 = prefetch.serve(stream.requests, store_path=os.path.join(scratch, "w4.bin"), window=4, **kw)
    assert s0.requests == s4.requests == 30
    assert s0.prefetch_reads == 0 and s0.on_demand_reads > 0
    assert s4.prefetch_hits > 0
    assert s4.on_demand_reads < s0.on_demand_reads
    assert s0.hit_tokens == s4.hit_tokens > 0     # the tiers change when bytes move, not what hits


def test_store_tasks_of_one_chunk_run_in_submission_order(scratch):
    """Writes, reads and writes of one chunk interleaved, with four I/O threads and
    other chunks' tasks in between: every read returns the write submitted just before
    it (never a torn mix), and the chunk ends with the last write."""
    cb = 256 * 1024
    st = pcr.ChunkStore(os.path.join(scratch, "order.bin"), cb, io_threads=4)
    versions = [np.full(cb, v, np.uint8) for v in range(1, 13)]
    others = [prefetch.chunk_pattern(50 + i, cb) for i in range(12)]
    reads = [np.zeros(cb, np.uint8) for _ in versions]
    for i, (w, o) in enumerate(zip(versions, others)):
        st.write_async(0, w)
        st.write_async(1 + i, o)
        st.read_async(0, reads[i])
    st.wait()
    for i, r in enumerate(reads):
        assert np.all(r == i + 1), f"read {i} saw a different or torn version"
    final = np.zeros(cb, np.uint8)
    st.read_async(0, final)
    st.wait()
    assert np.all(final == len(versions))
    back = [np.zeros(cb, np.uint8) for _ in others]
    for i, b in enumerate(back):
        st.read_async(1 + i, b)
    st.wait()
    assert all(np.array_equal(b, o) for b, o in zip(back, others))
    st.close()
