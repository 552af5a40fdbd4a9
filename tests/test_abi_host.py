"""C-ABI library on the CPU: it loads, exports every declared symbol, and its
host-side bookkeeping (admission against the page budget, page allocation,
page-table entries, placement) behaves as documented. A host-only pool
(device = -1) runs all of this without a GPU."""
import math
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS

HDR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "crosspool.h")
MLA16, MQA32, GQA = MODELS["mla16"], MODELS["mqa32"], MODELS["gqa32x4"]


def declared_functions():
    text = open(HDR).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cp_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(cpl.LIB, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", cpl._LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (cp_[a-z_0-9]+)", out))
    assert set(names) <= exported, set(names) - exported


def host_pool(pool_bytes=64 << 20, chunk=2 << 20, seed=0, max_requests=0):
    return cpl.Pool(page_tokens=64, pool_bytes=pool_bytes, chunk_bytes=chunk, placement_seed=seed, device=-1,
                    max_requests=max_requests)


def reg_all(p):
    return p.register_spec(MLA16), p.register_spec(MQA32), p.register_spec(GQA)


def test_model_geometry():
    p = host_pool()
    a, b, c = reg_all(p)
    ia, ib, ic = p.info(a), p.info(b), p.info(c)
    assert (ia["kappa"], ia["page_bytes"], ia["pages_per_chunk"], ia["d_k"], ia["d_v"]) == (1152, 73728, 28, 576, 512)
    assert (ib["kappa"], ib["page_bytes"], ib["pages_per_chunk"]) == (512, 32768, 64)
    assert (ic["kappa"], ic["page_bytes"], ic["pages_per_chunk"], ic["row_elems"]) == (2048, 131072, 16, 1024)
    p.destroy()


@pytest.mark.parametrize("kw,msg", [
    (dict(kind=cpl.CP_KIND_MLA, n_q_heads=16, n_kv_heads=2, latent_dim=512, rope_dim=64, softmax_scale=0.1), "exactly one"),
    (dict(kind=cpl.CP_KIND_MLA, n_q_heads=16, n_kv_heads=1, latent_dim=512, rope_dim=64), "softmax_scale"),
    (dict(kind=cpl.CP_KIND_GQA, n_q_heads=30, n_kv_heads=4, head_dim=128), "divide"),
    (dict(kind=cpl.CP_KIND_GQA, n_q_heads=32, n_kv_heads=4, head_dim=96), "V width"),
    (dict(kind=cpl.CP_KIND_GQA, n_q_heads=512, n_kv_heads=4, head_dim=128), "n_q_heads"),
    (dict(kind=7, n_q_heads=8, n_kv_heads=1, head_dim=128), "kind"),
])
def test_model_register_rejects_bad_geometry(kw, msg):
    p = host_pool()
    with pytest.raises(cpl.CrossPoolError) as e:
        cpl.cp_model_register(p.handle, **kw)
    assert e.value.status == cpl.CP_EINVAL and msg in e.value.message
    p.destroy()


def test_pool_create_validation():
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_pool_create(page_tokens=0, pool_bytes=1 << 20, device=-1)
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_pool_create(page_tokens=64, pool_bytes=1 << 20, chunk_bytes=2 << 20, device=-1)  # < one chunk
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_pool_create(page_tokens=64, pool_bytes=1 << 30, chunk_bytes=1000, device=-1)


def pte_to_chunk_slot(pte, chunk, page_bytes):
    off = int(pte) << 8
    return off // chunk, (off % chunk) // page_bytes, (off % chunk) % page_bytes


def test_page_tables_and_placement():
    chunk = 2 << 20
    p = host_pool(pool_bytes=64 * chunk, chunk=chunk, seed=0)
    a, b, c = reg_all(p)
    ra = p.open(a, 5000)
    rb = p.open(b, 3000)
    rc = p.open(c, 1000)
    p.append([ra, rb, rc], [4000, 3000, 1000], None)
    assert [p.ctx_len(r) for r in (ra, rb, rc)] == [4000, 3000, 1000]
    seen = {}
    for r, mid in ((ra, a), (rb, b), (rc, c)):
        pb = p.info(mid)["page_bytes"]
        ptes = p.pages(r)
        assert len(ptes) == math.ceil(p.ctx_len(r) / 64)
        for e in ptes:
            ch, slot, rem = pte_to_chunk_slot(e, chunk, pb)
            assert rem == 0 and ch < 64 and slot < chunk // pb
            assert seen.setdefault(ch, mid) == mid, "a chunk holds pages of one model only"
            assert (ch, slot) not in seen.get("slots", set())
            seen.setdefault("slots", set()).add((ch, slot))
    # seed 0: chunks handed out in ascending order, slots filled in order
    first = p.pages(ra)[:3]
    assert [pte_to_chunk_slot(e, chunk, 73728)[:2] for e in first] == [(0, 0), (0, 1), (0, 2)]
    for r in (ra, rb, rc):
        p.close(r)
    s = p.stats()
    assert s["chunks_used"] == 0 and s["pages_used"] == 0 and s["pages_reserved"] == 0 and s["requests_open"] == 0
    p.destroy()


def placement(seed):
    p = host_pool(pool_bytes=256 << 20, seed=seed)
    a, b, c = reg_all(p)
    rs = [p.open(a, 20000), p.open(c, 9000)]
    for _ in range(5):
        p.append(rs, [3000, 1500], None)
    out = [p.pages(r).copy() for r in rs]
    for r in rs:
        p.close(r)
    p.destroy()
    return out


def test_seeded_placement_is_reproducible_and_scattered():
    x1, x2, y = placement(7), placement(7), placement(8)
    assert all(np.array_equal(u, v) for u, v in zip(x1, x2))
    assert not all(np.array_equal(u, v) for u, v in zip(x1, y))
    chunks = np.array(x1[0], dtype=np.uint64) * 256 // (2 << 20)
    assert len(np.unique(chunks)) > 1 and not np.all(np.diff(chunks.astype(np.int64)) >= 0)


def test_admission_reject_changes_nothing():
    chunk = 2 << 20
    p = host_pool(pool_bytes=10 * chunk, chunk=chunk)
    a, b, c = reg_all(p)
    r1 = p.open(a, 64 * 28 * 6)  # six MLA chunks
    r2 = p.open(c, 64 * 16 * 3)  # three GQA chunks
    before = p.stats()
    with pytest.raises(cpl.CrossPoolError) as e:
        p.open(b, 64 * 64 * 2)  # two MQA chunks do not fit in the one left
    assert e.value.status == cpl.CP_ENOSPC
    assert p.stats() == before
    r3 = p.open(b, 64 * 64)  # exactly one chunk fits
    # admitted requests always get their pages, up to the reservation
    p.append([r1, r2, r3], [64 * 28 * 6, 64 * 16 * 3, 64 * 64], None)
    s = p.stats()
    assert s["chunks_used"] == 10 and s["pages_used"] == 28 * 6 + 16 * 3 + 64
    with pytest.raises(cpl.CrossPoolError) as e:
        p.open(a, 1)
    assert e.value.status == cpl.CP_ENOSPC
    p.close(r2)
    r4 = p.open(a, 64 * 28 * 3)
    p.append([r4], [64 * 28 * 3], None)
    for r in (r1, r3, r4):
        p.close(r)
    p.destroy()


def test_append_errors_are_atomic():
    p = host_pool()
    a, b, c = reg_all(p)
    r1, r2 = p.open(a, 100), p.open(b, 100)
    p.append([r1, r2], [10, 10], None)
    before = (p.stats(), p.ctx_len(r1), p.ctx_len(r2))
    for ids, nn in (([r1, r2], [10, 91]),  # past r2's reservation (2 pages = 128 tokens ok; 101 ok) -> use 200
                    ([r1, r1], [1, 1]), ([r1, 999], [1, 1]), ([r1], [-1])):
        if nn == [10, 91]:
            nn = [10, 200]
        with pytest.raises(cpl.CrossPoolError) as e:
            p.append(ids, nn, None)
        assert e.value.status == cpl.CP_EINVAL
        assert (p.stats(), p.ctx_len(r1), p.ctx_len(r2)) == before
    p.append([r1], [118], None)  # fills the reservation exactly (2 pages = 128 tokens)
    with pytest.raises(cpl.CrossPoolError):
        p.append([r1], [1], None)
    with pytest.raises(cpl.CrossPoolError) as e:
        p.decode([r1], 0, 0, 0)
    assert e.value.status == cpl.CP_ESTATE
    with pytest.raises(cpl.CrossPoolError) as e:
        p.gather(r1, 0, 1, 0)
    assert e.value.status == cpl.CP_ESTATE
    p.close(r1)
    with pytest.raises(cpl.CrossPoolError) as e:
        p.close(r1)
    assert e.value.status == cpl.CP_EINVAL
    with pytest.raises(cpl.CrossPoolError) as e:
        p.destroy()  # r2 still open
    assert e.value.status == cpl.CP_ESTATE
    p.close(r2)
    p.destroy()


def test_request_table_limit():
    p = host_pool(max_requests=3)
    a, _, _ = reg_all(p)
    ids = [p.open(a, 64) for _ in range(3)]
    with pytest.raises(cpl.CrossPoolError) as e:
        p.open(a, 64)
    assert e.value.status == cpl.CP_ENOSPC
    for r in ids:
        p.close(r)
    p.destroy()


def test_random_admission_never_strands_admitted_requests():
    """Random open / append / close traffic over three models. Whatever was
    admitted can always be filled to its full reservation, rejections change
    nothing, and pages are conserved."""
    rng = np.random.default_rng(123)
    chunk = 2 << 20
    p = host_pool(pool_bytes=24 * chunk, chunk=chunk, seed=99)
    mids = reg_all(p)
    live = {}
    for step in range(600):
        op = rng.integers(0, 3)
        if op == 0 or not live:
            m = int(rng.integers(0, 3))
            res = int(rng.integers(1, 6000))
            before = p.stats()
            try:
                r = p.open(mids[m], res)
                live[r] = res
            except cpl.CrossPoolError as e:
                assert e.status == cpl.CP_ENOSPC and p.stats() == before
        elif op == 1:
            r = int(rng.choice(list(live)))
            room = live[r] - p.ctx_len(r)
            if room > 0:
                p.append([r], [int(rng.integers(1, room + 1))], None)
        else:
            r = int(rng.choice(list(live)))
            p.close(r)
            del live[r]
        s = p.stats()
        assert s["chunks_used"] <= s["chunks_total"]
        assert s["pages_used"] == sum(math.ceil(p.ctx_len(r) / 64) for r in live)
    # fill every admitted request completely
    for r, res in live.items():
        room = res - p.ctx_len(r)
        if room:
            p.append([r], [room], None)
    for r in list(live):
        p.close(r)
    assert p.stats()["chunks_used"] == 0
    p.destroy()


# ---------------------------------------------------------------- virtual pools
# Host-only virtual pools run the same bookkeeping as device ones (address
# ranges per model, budget on mapped chunks) with the mapping calls left out.

def virtual_pool(pool_bytes=32 << 20, chunk=2 << 20, page_tokens=64, max_requests=0):
    return cpl.Pool(page_tokens=page_tokens, pool_bytes=pool_bytes, chunk_bytes=chunk, device=-1,
                    max_requests=max_requests, backing=cpl.CP_BACKING_VIRTUAL)


def test_virtual_pool_gives_each_model_its_own_range():
    chunk, n = 2 << 20, 16
    p = virtual_pool(pool_bytes=n * chunk, chunk=chunk)
    s = p.stats()
    assert s["backing"] == cpl.CP_BACKING_VIRTUAL and s["max_models"] == 16
    assert s["span_bytes"] == 16 * n * chunk
    mids = reg_all(p)
    lens = [3000, 2500, 900]
    rids = [p.open(m, L) for m, L in zip(mids, lens)]
    # admission maps the chunks of each whole reservation
    need = [math.ceil(math.ceil(L / 64) / p.info(m)["pages_per_chunk"]) for m, L in zip(mids, lens)]
    assert p.stats()["chunks_used"] == sum(need)
    p.append(rids, lens, None)
    assert p.stats()["chunks_used"] == sum(need)  # growth maps nothing
    for m, r, L, k in zip(mids, rids, lens, need):
        pb, ppc = p.info(m)["page_bytes"], p.info(m)["pages_per_chunk"]
        slots = set()
        for e in p.pages(r):
            ch, slot, rem = pte_to_chunk_slot(e, chunk, pb)
            assert rem == 0 and slot < ppc
            assert m * n <= ch < (m + 1) * n, "pages of model m lie in its own range"
            slots.add((ch, slot))
        assert len(slots) == math.ceil(L / 64)
        # a model's chunks fill its range from the bottom, slots in order
        assert sorted({c for c, _ in slots}) == list(range(m * n, m * n + k))
    p.close(rids[0])
    assert p.stats()["chunks_used"] == sum(need) - need[0]
    # a released slot is the first reused
    r = p.open(mids[0], 64)
    p.append([r], [1], None)
    assert pte_to_chunk_slot(p.pages(r)[0], chunk, p.info(mids[0])["page_bytes"])[:2] == (mids[0] * n, 0)
    for x in [r] + rids[1:]:
        p.close(x)
    assert p.stats()["chunks_used"] == 0
    p.destroy()


def test_virtual_pool_keeps_chunks_other_reservations_need():
    chunk = 2 << 20
    p = virtual_pool(pool_bytes=16 * chunk, chunk=chunk)
    a = p.register_spec(MLA16)
    ppc = p.info(a)["pages_per_chunk"]
    r1 = p.open(a, ppc * 64)        # one chunk
    r2 = p.open(a, ppc * 64 // 2)   # half a chunk: a second chunk
    assert p.stats()["chunks_used"] == 2
    p.append([r1, r2], [ppc * 64, 64], None)  # r1 fills chunk 0, r2 starts chunk 1
    p.close(r1)  # chunk 0 empties, but r2 is owed ppc/2 - 1 more pages: one chunk stays
    assert p.stats()["chunks_used"] == 1
    p.append([r2], [ppc * 64 // 2 - 64], None)  # grows into its reservation without mapping
    assert p.stats()["chunks_used"] == 1
    p.close(r2)
    assert p.stats()["chunks_used"] == 0
    p.destroy()


def test_virtual_pool_budget_caps_mapped_chunks():
    chunk = 2 << 20
    p = virtual_pool(pool_bytes=4 * chunk, chunk=chunk)
    a, b, c = reg_all(p)
    ppc_a = p.info(a)["pages_per_chunk"]
    ra = p.open(a, 3 * ppc_a * 64)  # three chunks of model a, mapped at admission
    assert p.stats()["chunks_used"] == 3
    before = p.stats()
    with pytest.raises(cpl.CrossPoolError) as e:
        p.open(c, 2 * p.info(c)["pages_per_chunk"] * 64)  # two more chunks: over the budget
    assert e.value.status == cpl.CP_ENOSPC and p.stats() == before
    rc = p.open(c, 64)
    assert p.stats()["chunks_used"] == 4 == p.stats()["chunks_total"]
    p.append([ra, rc], [3 * ppc_a * 64, 64], None)
    assert p.stats()["chunks_used"] == 4
    p.close(ra)
    assert p.stats()["chunks_used"] == 1
    p.close(rc)
    p.destroy()


def test_virtual_pool_model_count_follows_the_address_limit():
    # 256 GiB budget: four 256 GiB ranges fill the 1 TiB that page entries reach
    p = virtual_pool(pool_bytes=256 << 30, chunk=64 << 20, page_tokens=4096)
    assert p.stats()["max_models"] == 4
    for _ in range(4):
        p.register_spec(MQA32)
    with pytest.raises(cpl.CrossPoolError, match="address space for 4 models"):
        p.register_spec(MQA32)
    p.destroy()


def test_virtual_pool_create_validation():
    with pytest.raises(cpl.CrossPoolError, match="device_mem must be NULL"):
        cpl.Pool(page_tokens=64, pool_bytes=8 << 20, device=-1, device_mem=1 << 20, backing=cpl.CP_BACKING_VIRTUAL)
    with pytest.raises(cpl.CrossPoolError, match="unknown backing"):
        cpl.Pool(page_tokens=64, pool_bytes=8 << 20, device=-1, backing=7)


@pytest.mark.parametrize("backing", [cpl.CP_BACKING_BUFFER, cpl.CP_BACKING_VIRTUAL])
def test_random_traffic_invariants_both_backings(backing):
    """Open / append / close traffic: admitted requests always fill their
    reservations, rejections change nothing, mapped chunks never exceed the
    budget, and every chunk comes back at the end."""
    rng = np.random.default_rng(321)
    chunk = 2 << 20
    p = cpl.Pool(page_tokens=64, pool_bytes=20 * chunk, chunk_bytes=chunk, device=-1, placement_seed=5,
                 backing=backing)
    mids = reg_all(p)
    live = {}
    for step in range(500):
        op = rng.integers(0, 3)
        if op == 0 or not live:
            m = int(rng.integers(0, 3))
            before = p.stats()
            try:
                r = p.open(mids[m], int(rng.integers(1, 7000)))
                live[r] = (m, p.stats()["pages_reserved"] - before["pages_reserved"])
            except cpl.CrossPoolError as e:
                assert e.status == cpl.CP_ENOSPC and p.stats() == before
        elif op == 1:
            r = int(rng.choice(list(live)))
            room = live[r][1] * 64 - p.ctx_len(r)
            if room > 0:
                p.append([r], [int(rng.integers(1, room + 1))], None)
        else:
            r = int(rng.choice(list(live)))
            p.close(r)
            del live[r]
        s = p.stats()
        assert s["chunks_used"] <= s["chunks_total"]
        assert s["pages_used"] == sum(math.ceil(p.ctx_len(r) / 64) for r in live)
    for r, (m, pages) in live.items():
        room = pages * 64 - p.ctx_len(r)
        if room:
            p.append([r], [room], None)
    for r in list(live):
        p.close(r)
    assert p.stats()["chunks_used"] == 0
    p.destroy()


# ---------------------------------------------------------------- layer planes

def test_layer_planes_tables_and_budget():
    chunk = 2 << 20
    p = host_pool(pool_bytes=8 * chunk, chunk=chunk)
    a = p.register_spec(MLA16, n_layers=3)
    info = p.info(a)
    assert info["n_layers"] == 3
    ppc = info["pages_per_chunk"]
    r = p.open(a, ppc * 64)  # one chunk per plane
    assert p.stats()["pages_reserved"] == 3 * ppc
    p.append([r], [200], None)
    t = p.pages(r, layers=3)
    assert t.shape == (3, 4) and len(set(t.ravel().tolist())) == 12  # distinct pages in every plane
    assert p.stats()["pages_used"] == 12 and p.ctx_len(r) == 200
    assert p.cursor(r) == (0, 0)
    # the budget counts every plane: 3 of 8 chunks reserved, a second
    # request of two chunks per plane does not fit
    with pytest.raises(cpl.CrossPoolError) as e:
        p.open(a, 2 * ppc * 64)
    assert e.value.status == cpl.CP_ENOSPC
    r2 = p.open(a, ppc * 64 // 2)
    with pytest.raises(cpl.CrossPoolError):
        p.append([r2], [ppc * 64 // 2 + 1], None)  # past the reservation of each plane
    p.close(r)
    p.close(r2)
    assert p.stats()["chunks_used"] == 0 and p.stats()["pages_used"] == 0
    with pytest.raises(cpl.CrossPoolError, match="n_layers"):
        p.register_spec(MLA16, n_layers=1025)
    p.destroy()


def test_layer_planes_on_a_virtual_pool_map_every_plane_at_admission():
    chunk = 2 << 20
    p = virtual_pool(pool_bytes=16 * chunk, chunk=chunk)
    a = p.register_spec(MQA32, n_layers=4)
    ppc = p.info(a)["pages_per_chunk"]
    r = p.open(a, ppc * 64 + 1)  # two chunks' worth of pages per plane
    assert p.stats()["chunks_used"] == -(-4 * (ppc + 1) // ppc)
    p.append([r], [ppc * 64 + 1], None)
    assert p.stats()["chunks_used"] == -(-4 * (ppc + 1) // ppc)
    p.close(r)
    assert p.stats()["chunks_used"] == 0
    p.destroy()
