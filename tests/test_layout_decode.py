"""The kernel layouts the 16-bit conv kernels actually read, decoded on the
host back to dense weights and compared bit for bit with W * expand(mask)
(no GPU needed).

The canonical sections of a blob (Section 3 compact format) are checked
against the oracle's pack elsewhere; the kernels never read them.  They read
the derived sections, so these are decoded here:

* union / dense item layout: per wave tile and K-step, 8 item offsets (LDS
  byte offsets of a (4-channel block, kernel position) item) and the MFMA A
  operand in lane order [step][mfw][lane][8];
* pair layout (2:4 sparse MFMA): per step 16 item offsets, the kept 4x4
  weight blocks, and per (lane group, kernel group) a descriptor {block
  offset of its first pair, of its second pair, index register, 0}.

A decoded weight must land on a kept (filter, channel, position) exactly
once with the packed value, every kept weight must be found, and pruned
entries must be absent (union zero fill) -- so a dropped item, a duplicated
item, a wrong lane, a wrong channel or position decode, or a pair whose two
items share a kept group (one of them would be lost) all fail.
"""
import numpy as np
import pytest
import torch

from paper_2007_09835_amd import rt3d


@pytest.fixture(scope="module", autouse=True)
def built():
    from paper_2007_09835_amd import build
    build.build(force=False)


VAR_DENSE16, VAR_UNION16, VAR_PAIR16, VAR_BLOCKPAIR16 = 1, 3, 7, 8


def _bf16_bits(rng, shape, dt):
    w = rng.standard_normal(shape).astype(np.float32)
    if dt == "f16":
        return w.astype(np.float16).view(np.uint16)
    return torch.from_numpy(w).to(torch.bfloat16).view(torch.uint16).numpy()


def _plan(info):
    raw = bytes(info.plan)
    i32 = np.frombuffer(raw, dtype=np.int32)
    u64 = np.frombuffer(raw, dtype=np.uint64)
    t = dict(zip(("bt", "bh", "bw", "ht", "hh", "hw", "cc", "row", "slots", "nchunks"),
                 map(int, i32[:10])))
    t.update(mfw=int(i32[10]), wave_tiles=int(i32[11]), ips=int(i32[12]),
             tile_steps=int(i32[13]), gmap=int(i32[14]), step_ptr=int(u64[8]),
             item_ptr=int(u64[9]), items=int(u64[10]), a=int(u64[11]), keep=int(u64[12]))
    return t


def _item(p, off, kh, kw):
    """(channel block within the chunk, kernel position) of an LDS offset."""
    row, es = p["row"], 2
    ql = (off % row) // (4 * es)
    r = off // row
    iw = r % p["hw"]
    ih = (r // p["hw"]) % p["hh"]
    it = r // (p["hw"] * p["hh"])
    assert iw < kw and ih < kh, (off, iw, ih)
    return ql, (it * kh + ih) * kw + iw


def _u32(blob, off, count):
    return np.frombuffer(blob[off:off + 4 * count].tobytes(), dtype=np.uint32)


def decode(desc, info, blob):
    """Dense [M][N][K_s] uint16 image of the derived layout, and the number
    of weight slots the layout streams (zero fill included)."""
    p = _plan(info)
    M, N, kt, kh, kw = desc.c_out, desc.c_in, desc.kt, desc.kh, desc.kw
    ks = kt * kh * kw
    out = np.zeros((M, N, ks), dtype=np.uint16)
    seen = np.zeros((M, N, ks), dtype=bool)
    nwt, nch, cc = p["wave_tiles"], p["nchunks"], p["cc"]
    step_ptr = _u32(blob, p["step_ptr"], nwt * (nch + 1)).reshape(nwt, nch + 1)
    item_ptr = _u32(blob, p["item_ptr"], nwt)
    a16 = np.frombuffer(blob[p["a"]:].tobytes()[: (len(blob) - p["a"]) // 2 * 2], dtype=np.uint16)
    streamed = 0

    def put(m, c, pos, v):
        if m >= M or c >= N:
            assert v == 0, ("padding row/column holds a weight", m, c)
            return
        if v == 0:
            return
        assert not seen[m, c, pos], ("weight streamed twice", m, c, pos)
        seen[m, c, pos] = True
        out[m, c, pos] = v

    if info.variant == VAR_BLOCKPAIR16:
        idx_all = _u32(blob, p["keep"], (p["a"] - p["keep"]) // 4)
        for wt in range(nwt):
            for ch in range(nch):
                for s in range(step_ptr[wt, ch], step_ptr[wt, ch + 1]):
                    its = _u32(blob, p["items"] + 32 * s, 8)
                    for lane in range(64):
                        m = wt * 16 + (lane & 15)
                        idx = int(idx_all[s * 64 + lane])
                        for h in range(2):
                            j = 2 * (lane >> 4) + h           # slot of this A half
                            off = int(its[2 * (j % 4) + j // 4])
                            ql, pos = _item(p, off, kh, kw)
                            assert ql % 2 == 0, "block pairs start at an even channel block"
                            sel = (idx >> (8 * h)) & 0xFF
                            assert sel in (0x44, 0xEE), hex(sel)
                            ql += 1 if sel == 0xEE else 0
                            for c in range(4):
                                streamed += 1
                                put(m, 4 * (ch * (cc // 4) + ql) + c, pos,
                                    int(a16[(s * 64 + lane) * 8 + 4 * h + c]))
        return out, seen, streamed

    if info.variant == VAR_PAIR16 and p["mfw"] > 1:
        mfw = p["mfw"]
        idx_all = _u32(blob, p["keep"], (p["a"] - p["keep"]) // 4)
        for wt in range(nwt):
            for ch in range(nch):
                for s in range(step_ptr[wt, ch], step_ptr[wt, ch + 1]):
                    its = _u32(blob, p["items"] + 64 * s, 16)
                    for i in range(mfw):
                        base = (s * mfw + i) * 64
                        for lane in range(64):
                            m = wt * 16 * mfw + 16 * i + (lane & 15)
                            idx = int(idx_all[base + lane])
                            for h in range(2):
                                j = 2 * (lane >> 4) + h
                                lg, half = j % 4, (j // 4) * 2
                                sel = (idx >> (8 * h)) & 0xFF
                                assert sel in (0x44, 0xEE), hex(sel)
                                off = int(its[4 * lg + half + (1 if sel == 0xEE else 0)])
                                ql, pos = _item(p, off, kh, kw)
                                for c in range(4):
                                    streamed += 1
                                    put(m, 4 * (ch * (cc // 4) + ql) + c, pos,
                                        int(a16[(base + lane) * 8 + 4 * h + c]))
        return out, seen, streamed

    if info.variant == VAR_PAIR16:
        used_blocks = set()
        for wt in range(nwt):
            for ch in range(nch):
                for s in range(step_ptr[wt, ch], step_ptr[wt, ch + 1]):
                    its = _u32(blob, p["items"] + 64 * s, 16)
                    desc = _u32(blob, p["keep"] + 256 * s, 64).reshape(4, 4, 4)  # [g][group]
                    for j in range(8):
                        lg, half = j % 4, (j // 4) * 2
                        x_off, y_off = int(its[4 * lg + half]), int(its[4 * lg + half + 1])
                        for gi in range(4):
                            # A side: lane group j // 2 holds pair j in its half j % 2
                            d = desc[j // 2, gi]
                            boff, idx = int(d[j % 2]), (int(d[2]) >> (8 * (j % 2))) & 0xFF
                            if boff >= 1 << 31:
                                continue
                            assert idx in (0x44, 0xEE), hex(idx)
                            assert boff % 32 == 0
                            off = y_off if idx == 0xEE else x_off
                            ql, pos = _item(p, off, kh, kw)
                            blk = boff // 32
                            assert blk not in used_blocks, "block referenced twice"
                            used_blocks.add(blk)
                            streamed += 16
                            for r in range(4):
                                for c in range(4):
                                    put(16 * wt + 4 * gi + r, 4 * (ch * (cc // 4) + ql) + c, pos,
                                        int(a16[16 * blk + 4 * r + c]))
        return out, seen, streamed

    mfw = p["mfw"]
    items = _u32(blob, p["items"], (len(blob) - p["items"]) // 4)
    dense = info.variant == VAR_DENSE16
    # Union layouts may reorder the 4-filter blocks: the keep section then
    # holds the layer block of every wave-tile block slot.
    gmap = None
    if p["gmap"]:
        assert info.variant == VAR_UNION16
        gmap = _u32(blob, p["keep"], nwt * 4 * mfw)
        real = [int(b) for b in gmap if b < (M + 3) // 4]
        assert sorted(real) == list(range((M + 3) // 4)), "block map is not a permutation"
    for wt in range(nwt):
        row0, step0 = int(item_ptr[wt]), int(step_ptr[wt, 0])
        for ch in range(nch):
            for s in range(step_ptr[wt, ch], step_ptr[wt, ch + 1]):
                its = items[(row0 + s - step0) * 8:(row0 + s - step0) * 8 + 8]
                for i in range(mfw):
                    base = (s * mfw + i) * 64 * 8
                    for lane in range(64):
                        m = wt * 16 * mfw + 16 * i + (lane & 15)
                        if gmap is not None:
                            m = 4 * int(gmap[m // 4]) + m % 4
                        for e in range(8):
                            ql, pos = _item(p, int(its[2 * (lane >> 4) + e // 4]), kh, kw)
                            streamed += 1
                            put(m, 4 * (ch * (cc // 4) + ql) + e % 4, pos, int(a16[base + lane * 8 + e]))
        if dense:
            assert row0 == 0
    return out, seen, streamed


def expected(w_bits, mask, g):
    M, N = w_bits.shape[:2]
    full = np.repeat(np.repeat(mask, g[0], 0), g[1], 1)[:M, :N]
    return np.where(full == 1, w_bits.reshape(M, N, -1), 0).astype(np.uint16), full == 1


CASES = [
    # c_in, c_out, thw, k, stride, pad, g, keep, n
    (32, 48, (4, 7, 9), (3, 3, 3), (1, 1, 1), (1, 1, 1), (4, 4), 9, 1),
    (24, 20, (5, 7, 6), (3, 3, 3), (2, 2, 2), (1, 1, 1), (4, 4), 12, 2),
    (10, 13, (3, 9, 11), (3, 3, 3), (1, 1, 1), (1, 1, 1), (4, 4), 7, 1),    # partial groups
    (40, 36, (6, 5, 5), (3, 1, 1), (2, 1, 1), (1, 0, 0), (4, 4), 2, 1),
    (64, 64, (4, 8, 8), (1, 3, 3), (1, 1, 1), (0, 1, 1), (8, 4), 4, 1),
    (128, 64, (4, 6, 6), (3, 3, 3), (1, 1, 1), (1, 1, 1), (4, 4), 27, 1),   # all kept: no pairs
    (48, 32, (3, 6, 6), (3, 3, 3), (1, 1, 1), (1, 1, 1), (4, 4), 0, 1),     # nothing kept
]


def _mask(rng, c_out, c_in, ks, g, keep):
    P, Q = -(-c_out // g[0]), -(-c_in // g[1])
    m = np.zeros((P, Q, ks), np.uint8)
    for p in range(P):
        for q in range(Q):
            m[p, q, rng.choice(ks, keep, replace=False)] = 1
    return m


@pytest.mark.parametrize("tune", ["kgs_map=2", "kgs_map=1", "kgs_map=1,pair_mfw=2", "kgs_map=1,pair_mfw=4",
                                  "kgs_map=0,kgs_mfw=1", "kgs_map=0,kgs_mfw=2",
                                  "kgs_map=0,kgs_mfw=4", "kgs_map=0,kgs_mfw=1,slots=128"])
@pytest.mark.parametrize("ci", range(len(CASES)))
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_kgs_layout_decodes_to_masked_weights(dt, ci, tune, monkeypatch):
    monkeypatch.setenv("RT3D_TUNE", tune)
    c_in, c_out, thw, k, stride, pad, g, keep, n = CASES[ci]
    rng = np.random.default_rng(40 + ci)
    w = _bf16_bits(rng, (c_out, c_in, *k), dt)
    ks = k[0] * k[1] * k[2]
    mask = _mask(rng, c_out, c_in, ks, g, keep)
    desc = rt3d.make_desc(n, c_in, c_out, thw, k, stride, pad, g, dt)
    blob, info = rt3d.rt3d_kgs_pack(desc, w, mask)
    want_pair = tune.startswith("kgs_map=1")
    want = {"kgs_map=1": VAR_PAIR16, "kgs_map=2": VAR_BLOCKPAIR16}.get(tune.split(",")[0], VAR_UNION16)
    assert info.variant == want, info.variant
    got, seen, streamed = decode(desc, info, blob)
    exp, kept = expected(w, mask, g)
    assert got.tobytes() == exp.tobytes()
    # every kept nonzero weight was found (random normal weights are nonzero)
    assert np.array_equal(seen, kept & (exp != 0))
    if want_pair and "pair_mfw" not in tune:
        # kept 4x4 blocks only: the stream is the canonical values' size
        # (partial trailing groups stream their zero rows and columns)
        if c_out % 4 == 0 and c_in % 4 == 0:
            assert streamed == info.kept_weights
        else:
            assert info.kept_weights <= streamed < info.kept_weights + 16 * mask.sum() * 4


@pytest.mark.parametrize("mfw", ["1", "2", "4"])
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_dense_layout_decodes_to_weights(dt, mfw, monkeypatch):
    monkeypatch.setenv("RT3D_TUNE", "dense_mfw=" + mfw)
    rng = np.random.default_rng(7)
    c_in, c_out = 40, 72
    w = _bf16_bits(rng, (c_out, c_in, 3, 3, 3), dt)
    desc = rt3d.make_desc(1, c_in, c_out, (4, 8, 9), dtype=dt)
    blob, info = rt3d.rt3d_dense_pack(desc, w)
    assert info.variant == VAR_DENSE16
    got, seen, _ = decode(desc, info, blob)
    assert got.tobytes() == w.reshape(c_out, c_in, 27).tobytes()
    assert seen.all()


def test_pair_stream_is_the_kept_weights_for_c3d_layers(monkeypatch):
    """For the C3D conv stack's KGS layers at about 3x (4x4 groups), the pair
    layout streams exactly the kept 4x4 blocks: its weight section is the
    canonical values' size (plus section alignment)."""
    from paper_2007_09835_amd import synth
    monkeypatch.setenv("RT3D_TUNE", "kgs_map=1")
    for l in synth.c3d_stack(3.0):
        if l.dense:
            continue
        d = synth.layer_params("c3d", l, mask_kind="kgs", rate=3.0)
        desc = rt3d.make_desc(1, l.c_in, l.c_out, (l.t, l.h, l.w), l.k, l.stride, l.pad, l.g,
                              "bf16", pool=l.pool_after[0] if l.pool_after else (1, 1, 1))
        blob, info = rt3d.rt3d_kgs_pack(desc, synth.to_dtype(d.w, "bf16"), d.mask)
        assert info.variant == VAR_PAIR16
        p = _plan(info)
        a_bytes = info.packed_bytes - p["a"]
        assert a_bytes <= info.canon_bytes[3] + 255, (l.name, a_bytes, info.canon_bytes[3])


# ---------------------------------------------------------------------------
# Randomised shapes: group sizes, partial groups, strides, paddings, kernel
# extents and kept counts drawn by hypothesis, every mapping decoded.
# ---------------------------------------------------------------------------

from hypothesis import HealthCheck, given, settings, strategies as st  # noqa: E402

MAPPINGS = ["kgs_map=0,kgs_mfw=1", "kgs_map=0,kgs_mfw=2", "kgs_map=0,kgs_mfw=4", "kgs_map=1",
            "kgs_map=1,pair_mfw=2", "kgs_map=1,pair_mfw=4", "kgs_map=2",
            "kgs_map=0,kgs_mfw=1,kgs_order=1", "kgs_map=0,kgs_mfw=2,kgs_order=1"]


@st.composite
def _layer(draw):
    g = draw(st.sampled_from([(4, 4), (8, 4), (16, 4), (4, 8), (16, 8)]))
    c_in = draw(st.integers(5, 72))
    c_out = draw(st.integers(1, 80))
    k = draw(st.sampled_from([(3, 3, 3), (1, 3, 3), (3, 1, 1), (1, 1, 1), (1, 5, 5)]))
    stride = draw(st.sampled_from([(1, 1, 1), (2, 2, 2), (1, 2, 2)]))
    pad = tuple(kk // 2 for kk in k)
    thw = (draw(st.integers(k[0], 6)), draw(st.integers(k[1], 9)), draw(st.integers(k[2], 9)))
    ks = k[0] * k[1] * k[2]
    keep = draw(st.integers(0, ks))
    return c_in, c_out, thw, k, stride, pad, g, keep


@settings(max_examples=80, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(case=_layer(), tune=st.sampled_from(MAPPINGS), dt=st.sampled_from(["bf16", "f16"]),
       seed=st.integers(0, 2**31 - 1))
def test_random_layers_decode_to_masked_weights(case, tune, dt, seed, monkeypatch):
    monkeypatch.setenv("RT3D_TUNE", tune)
    c_in, c_out, thw, k, stride, pad, g, keep = case
    rng = np.random.default_rng(seed)
    w = _bf16_bits(rng, (c_out, c_in, *k), dt)
    mask = _mask(rng, c_out, c_in, k[0] * k[1] * k[2], g, keep)
    desc = rt3d.make_desc(1, c_in, c_out, thw, k, stride, pad, g, dt)
    blob, info = rt3d.rt3d_kgs_pack(desc, w, mask)
    got, seen, _ = decode(desc, info, blob)
    exp, kept = expected(w, mask, g)
    assert got.tobytes() == exp.tobytes()
    assert np.array_equal(seen, kept & (exp != 0))


@pytest.mark.parametrize("mfw", ["1", "2"])
def test_union_reorders_blocks_that_keep_alike(mfw, monkeypatch):
    """Blocks 0, 2, 4, ... keep one item set and blocks 1, 3, 5, ... a
    disjoint one: in layer order every wave tile multiplies both sets, so the
    planner must put alike blocks together (a block map in the keep
    section), shrink the K-steps to one set's worth, and the layout must
    still decode to W * expand(mask); with reordering switched off the steps
    are the union of both sets."""
    c_in, c_out, k = 32, 64, (3, 3, 3)
    ks = 27
    rng = np.random.default_rng(5)
    w = _bf16_bits(rng, (c_out, c_in, *k), "bf16")
    P, Q = c_out // 4, c_in // 4
    mask = np.zeros((P, Q, ks), np.uint8)
    mask[0::2, :, 0:9] = 1
    mask[1::2, :, 9:18] = 1
    desc = rt3d.make_desc(1, c_in, c_out, (4, 6, 6), k, (1, 1, 1), (1, 1, 1), (4, 4), "bf16")
    steps = {}
    for order in ("1", "0"):
        monkeypatch.setenv("RT3D_TUNE", "kgs_map=0,kgs_mfw=%s,kgs_order=%s" % (mfw, order))
        blob, info = rt3d.rt3d_kgs_pack(desc, w, mask)
        assert info.variant == VAR_UNION16
        p = _plan(info)
        assert p["gmap"] == (1 if order == "1" else 0)
        got, _, _ = decode(desc, info, blob)
        exp, _ = expected(w, mask, (4, 4))
        assert got.tobytes() == exp.tobytes()
        nwt, nch = p["wave_tiles"], p["nchunks"]
        sp = _u32(blob, p["step_ptr"], nwt * (nch + 1)).reshape(nwt, nch + 1)
        steps[order] = int((sp[:, nch] - sp[:, 0]).sum())
    # 8 channel blocks x 9 positions per set: 9 steps per tile and chunk
    # when alike blocks share a tile, 18 when each tile mixes both sets.
    assert steps["1"] * 2 == steps["0"], steps
