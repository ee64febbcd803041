"""GPU tests of the streaming-pattern probe (a measurement tool, no operation
of the paper): streams read and written in place and streams only read keep
their bits; streams only written receive stream 0's words (their upper
halves for 2-byte streams), or the run index when no stream is read; the
elements a shape skips (the last n mod 4, or everything past the last whole
tile) are untouched; the reported bytes count every read and write; patterns
that are not instantiated, out-of-order classes and bad buffers launch
nothing."""
import numpy as np
import pytest
import torch

import paper_2609_36662_amd as al

pytestmark = pytest.mark.gpu

R, W, RW = al.PROBE_READ, al.PROBE_WRITE, al.PROBE_READ | al.PROBE_WRITE
TILE = 4 * 4 * 256          # elements of one tile per stream (4 runs of 4 per lane, 256 lanes)
RUNS = (al.PROBE_RUN1, al.PROBE_RUN2, al.PROBE_RUN8)
TILES = (al.PROBE_SERIAL, al.PROBE_TILE)


@pytest.fixture(scope="module")
def ctx():
    c = al.autoloco_create(0)
    yield c
    c.close()


def _bufs(n, count, seed, dtype=torch.float32):
    g = torch.Generator().manual_seed(seed)
    return [torch.randn(n, generator=g).to(dtype).cuda() for _ in range(count)]


def _bits(t):
    t = t.detach().cpu()
    return t.view(torch.int16).numpy().copy() if t.element_size() == 2 else t.view(torch.int32).numpy().copy()


def _moved(shape, n):
    return n // TILE * TILE if shape in TILES else n // 4 * 4


SIZES = [5, 4 * 256 + 3, 3 * TILE + 1000, 256 * 4 * 9 + 2, 8 * 1024 * 7 + 3 * 1024 + 3]


@pytest.mark.parametrize("shape", RUNS + TILES)
@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("blocks", [0, 3])
@pytest.mark.parametrize("access", [RW, R])
def test_in_place_and_read_streams_keep_their_bits(ctx, shape, n, blocks, access):
    bufs = _bufs(n, 10, seed=n + shape)
    before = [_bits(b) for b in bufs]
    moved = al.autoloco_traffic_probe(ctx, [(b, access) for b in bufs], shape, blocks)
    torch.cuda.synchronize()
    for i, b in enumerate(bufs):
        assert np.array_equal(_bits(b), before[i]), f"stream {i} changed"
    assert moved == 4.0 * _moved(shape, n) * 10 * (2 if access == RW else 1)


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("shape,k", [(al.PROBE_RUN1, 1), (al.PROBE_RUN1, 2), (al.PROBE_RUN1, 4), (al.PROBE_RUN1, 8), (al.PROBE_RUN1, 16),
                                     (al.PROBE_RUN8, 4), (al.PROBE_RUN8, 8), (al.PROBE_RUN8, 16)])
def test_written_streams_receive_stream_0(ctx, n, shape, k):
    # the reset's pattern: theta read, k streams written with its words
    bufs = _bufs(n, k + 1, seed=3 * n + k)
    before = [_bits(b) for b in bufs]
    moved = al.autoloco_traffic_probe(ctx, [(bufs[0], R)] + [(b, W) for b in bufs[1:]], shape, 3)
    torch.cuda.synchronize()
    per = n // 4 * 4
    for i in range(1, k + 1):
        got = _bits(bufs[i])
        assert np.array_equal(got[:per], before[0][:per])
        assert np.array_equal(got[per:], before[i][per:])      # skipped elements untouched
    assert np.array_equal(_bits(bufs[0]), before[0])
    assert moved == 4.0 * per * (k + 1)


@pytest.mark.parametrize("n", SIZES)
def test_two_byte_streams(ctx, n):
    # the shard step's pattern: theta and v in place, 8 two-byte streams read, one written
    th, v = _bufs(n, 2, seed=11)
    recv = _bufs(n, 8, seed=12, dtype=torch.bfloat16)
    (mean,) = _bufs(n, 1, seed=13, dtype=torch.bfloat16)
    b = [_bits(x) for x in [th, v] + recv]
    b_mean = _bits(mean)
    moved = al.autoloco_traffic_probe(ctx, [(th, RW), (v, RW)] + [(r, R) for r in recv] + [(mean, W)],
                                      al.PROBE_RUN2, 0)
    torch.cuda.synchronize()
    per = n // 4 * 4
    for x, old in zip([th, v] + recv, b):
        assert np.array_equal(_bits(x), old)
    upper = (b[0].view(np.uint32) >> 16).astype(np.uint16).view(np.int16)
    got = _bits(mean)
    assert np.array_equal(got[:per], upper[:per])
    assert np.array_equal(got[per:], b_mean[per:])
    assert moved == per * (2 * 4 * 2 + 8 * 2 + 2)


@pytest.mark.parametrize("shape", [al.PROBE_RUN1, al.PROBE_RUN8, al.PROBE_TILE, al.PROBE_SERIAL])
def test_pure_write_writes_run_index(ctx, shape):
    n = 3 * TILE + 7
    bufs = _bufs(n, 10, seed=5)
    al.autoloco_traffic_probe(ctx, [(b, W) for b in bufs], shape, 0)
    torch.cuda.synchronize()
    per = _moved(shape, n)
    want = np.repeat(np.arange(per // 4, dtype=np.int32), 4)
    for b in bufs:
        assert np.array_equal(_bits(b)[:per], want)


def test_bad_arguments_launch_nothing(ctx):
    bufs = _bufs(4096, 12, seed=1)
    half = _bufs(4096, 2, seed=2, dtype=torch.bfloat16)
    before = [_bits(b) for b in bufs + half]
    bad = [
        ([(b, RW) for b in bufs[:11]], al.PROBE_RUN1, 0),            # 11 in place: not instantiated
        ([(b, RW) for b in bufs[:4]], al.PROBE_SERIAL, 0),           # tiles take 10 streams
        ([(bufs[0], W), (bufs[1], R)], al.PROBE_RUN1, 0),            # classes out of order
        ([(half[0], RW)], al.PROBE_RUN2, 0),                         # 2-byte stream in place
        ([(bufs[0], 0)], al.PROBE_RUN1, 0),                          # no access
        ([(bufs[0], R), (bufs[1], W)], al.PROBE_RUN8, 0),            # 1 read, 1 written: not at 8 runs
        ([(bufs[0], RW)], 7, 0),                                     # unknown shape
        ([(bufs[0], RW)], al.PROBE_RUN1, 20000),                     # too many workgroups
    ]
    for spec, shape, blocks in bad:
        with pytest.raises(al.AutolocoError) as e:
            al.autoloco_traffic_probe(ctx, spec, shape, blocks)
        assert e.value.status == -1
    with pytest.raises(al.AutolocoError) as e:                       # overlapping streams
        al.autoloco_traffic_probe(ctx, [(bufs[0], RW), (bufs[0][4:], RW)], al.PROBE_RUN1, 0, n=4000)
    assert e.value.status == -3
    with pytest.raises(al.AutolocoError) as e:                       # misaligned stream
        al.autoloco_traffic_probe(ctx, [(bufs[0], RW), (bufs[1][1:], RW)], al.PROBE_RUN1, 0, n=4000)
    assert e.value.status == -2
    torch.cuda.synchronize()
    for i, b in enumerate(bufs + half):
        assert np.array_equal(_bits(b), before[i])


PHASE_TILE = 7 * 4 * 256      # elements of one phased tile per stream


@pytest.mark.parametrize("blocks", [1, 3, 0])
def test_phased_keeps_bits_and_counts_whole_rounds(ctx, blocks):
    grid = blocks or torch.cuda.get_device_properties(0).multi_processor_count
    n = 2 * grid * PHASE_TILE + 1000 if blocks else grid * PHASE_TILE + 77
    bufs = _bufs(n, 10, seed=blocks + 40)
    before = [_bits(b) for b in bufs]
    moved = al.autoloco_traffic_probe(ctx, [(b, RW) for b in bufs], al.PROBE_PHASED, blocks)
    torch.cuda.synchronize()
    for i, b in enumerate(bufs):
        assert np.array_equal(_bits(b), before[i]), f"stream {i} changed"
    assert moved == 4.0 * (n // (grid * PHASE_TILE)) * grid * PHASE_TILE * 10 * 2


def test_phased_rejects_other_patterns(ctx):
    bufs = _bufs(PHASE_TILE, 10, seed=9)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    for spec, blocks in (([(b, RW) for b in bufs[:9]], 1),          # nine streams
                         ([(b, R) for b in bufs], 1),               # read only
                         ([(b, RW) for b in bufs], 2 * cus + 1)):   # more workgroups than fit at once
        with pytest.raises(al.AutolocoError) as e:
            al.autoloco_traffic_probe(ctx, spec, al.PROBE_PHASED, blocks)
        assert e.value.status == -1
