"""Two replica processes share one pool through a tier process (the paper's shared host tier,
Sec. 2 and Fig. 1), with the host-side completion handshake of Sec. 3.2.

Three processes on the GPU: the tier owns the pinned pool; replica A (a child process) stores
its prefix through the tier; replica B (this test) loads it into a fresh fragmented block set.
The pool bytes (dumped by the tier) and B's cache are compared with the oracle.
"""
import contextlib
import gc
import os
import signal
import socket
import struct
import subprocess
import sys
import time

import numpy as np
import pytest
import torch

import harness
from paper_2609_15021_amd import kvx
from tests.gpu_support import DEV, TINY, TORCH_INT, first_mismatch, host_cache, oracle_pool, oracle_unpack_into

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _fresh_segments():
    """Buffers shared with the tier must be their own allocations under 2 GiB: release the caching
    allocator's free segments first (earlier tests leave huge ones that small tensors would be
    carved from, and kv_ipc_export rightly refuses to share those)."""
    gc.collect()  # tensors held only by reference cycles (e.g. a caught exception's frames) go first
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    yield

ROLES = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tier_roles.py")
POOL_SENT = 0xA5


def _dims(lay):
    return [str(v) for v in (lay.L, lay.H, lay.D, lay.E, lay.BS, lay.C)]


def _start_tier(sock, lay, slots, mode, nconn, dump, role="tier", extra=()):
    p = subprocess.Popen([sys.executable, "-u", ROLES, role, sock, *_dims(lay), str(slots), mode, str(nconn), dump,
                          *extra], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    t0 = time.time()
    while time.time() - t0 < 90:
        line = p.stdout.readline()
        if line.startswith("READY"):
            return p
        if not line and p.poll() is not None:
            break
    p.kill()
    raise AssertionError(f"tier did not start: {p.stdout.read()[-2000:]}")


def _finish_tier(p):
    out, _ = p.communicate(timeout=90)
    assert p.returncode == 0, out[-2000:]
    line = [ln for ln in out.splitlines() if ln.startswith("TIER")][-1]
    assert set(line.split(" ", 1)[1].split(";")) == {"ok"}, line


def _store_process(sock, lay, NB, n, seed, delay_ms):
    r = subprocess.run([sys.executable, "-u", ROLES, "store", sock, *_dims(lay), str(NB), str(n), str(seed),
                        str(delay_ms)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "STORED" in r.stdout, (r.stdout + r.stderr)[-3000:]


def _connect(sock):
    c = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    c.connect(sock)
    _OPEN.append(c)
    return c


_OPEN = []  # sockets of the running test, closed if it fails


@contextlib.contextmanager
def _serving(tier):
    """Run a test body against a started tier: on any failure close the test's sockets and kill
    the tier, so the original error surfaces instead of a wait for connections that never come."""
    _OPEN.clear()
    try:
        yield tier
    except BaseException:
        for c in _OPEN:
            c.close()
        tier.kill()
        out, _ = tier.communicate(timeout=30)
        print("tier output:", (out or "")[-3000:])  # shown by pytest with the failure
        raise


@pytest.mark.parametrize("mode", ["zero_copy", "staged", "staged+zero_copy"])
def test_two_replica_processes_share_one_pool(mode, tmp_path):
    lay = TINY
    n = 3 * lay.C + 100
    nc, NB = lay.nc(n), lay.nblk(n) + 9
    seed = harness.sub_seed("tier", mode)
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_tier(sock, lay, nc + 2, mode, 2, dump)
    with _serving(tier):
        _store_process(sock, lay, NB, n, seed, 0)
        btB = harness.block_table(seed + 2, NB, lay.nblk(n))
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        s = torch.cuda.Stream()
        torch.cuda.synchronize()
        c = _connect(sock)
        kvx.kv_tier_load(c.fileno(), kvx.Cache(dB, lay.kv, NB), btB, n, np.arange(nc), s)
        got_B = dB.cpu()  # the load completed before kv_tier_load returned
        c.close()
    _finish_tier(tier)
    A = host_cache(lay, NB, seed, "raw")
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    want_pool = oracle_pool(lay, A, btA, n, np.arange(nc), nc + 2, POOL_SENT)
    pool = np.load(dump)
    assert np.array_equal(pool, want_pool), first_mismatch(pool, want_pool)
    want_B = oracle_unpack_into(lay, np.zeros_like(A), btB, n, want_pool, np.arange(nc))
    got = got_B.numpy().view(A.dtype).reshape(A.shape)
    assert np.array_equal(got, want_B), first_mismatch(got, want_B)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_delayed_producer_across_processes(mode, tmp_path):
    """Replica A's producer writes byte 37 after a 60 ms spin on its stream; the store request
    leaves A only after that stream completed, so every committed byte is 37 (Sec. 3.2)."""
    lay = TINY
    n = 1024
    nc, NB = lay.nc(n), lay.nblk(n) + 4
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_tier(sock, lay, nc, mode, 1, dump)
    with _serving(tier):
        _store_process(sock, lay, NB, n, harness.sub_seed("tier-37", mode), 60)
    _finish_tier(tier)
    pool = np.load(dump)
    assert pool.size == nc * lay.slot_bytes and (pool == 37).all()


def test_tier_rejects_a_bad_request_and_keeps_serving(tmp_path):
    lay = TINY
    n = 512
    nc, NB = lay.nc(n), 64
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_tier(sock, lay, nc, "staged", 1, dump)
    with _serving(tier):
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        cache = kvx.Cache(dB, lay.kv, NB)
        bt = np.arange(lay.nblk(n), dtype=np.int32)
        c = _connect(sock)
        with pytest.raises(kvx.KvError) as e:
            kvx.kv_tier_load(c.fileno(), cache, bt, n, [0, nc], None)   # chunk id outside the pool
        assert e.value.status == kvx.KV_EINVAL and "tier:" in str(e.value)
        big = kvx.Cache(dB, lay.kv, NB)
        big.struct.num_blocks = 10000                                 # claims more than B's allocation
        with pytest.raises(kvx.KvError) as e:
            kvx.kv_tier_load(c.fileno(), big, bt, n, np.arange(nc), None)
        assert e.value.status == kvx.KV_EINVAL and "exceeds its shared allocation" in str(e.value)
        kvx.kv_tier_load(c.fileno(), cache, bt, n, np.arange(nc), None)  # still served
        c.close()
    _finish_tier(tier)


def test_ipc_export_refuses_allocations_of_2_gib():
    t = torch.empty(2 << 30, dtype=torch.uint8, device=DEV)
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_ipc_export(t)
    status = e.value.status
    # The caught exception's traceback holds the frames that reference t (a reference cycle):
    # drop it and collect, or the 2 GiB segment outlives the test and later small tensors are
    # carved from it.
    del e
    assert status == kvx.KV_EUNSUPPORTED
    small = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    buf = kvx.kv_ipc_export(small[4096:])
    assert buf.allocation_bytes < (2 << 30) and buf.offset >= 4096
    del t, small
    gc.collect()
    torch.cuda.empty_cache()


def test_tier_survives_a_malformed_connection(tmp_path):
    """A connection that sends a garbage frame ends with an error on its own, and so does one whose
    header announces a block table of 2^62 entries (sizes that would overflow the payload arithmetic);
    the tier keeps serving the next replica."""
    lay = TINY
    n = 512
    nc, NB = lay.nc(n), 64
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    p = _start_tier(sock, lay, nc, "staged", 3, dump)
    with _serving(p):
        bad = _connect(sock)
        bad.sendall(b"\x00" * 160)  # a full header's worth of bytes with the wrong magic
        bad.close()
        # A well-formed load header (magic "KVXT", op 2) with an absurd table length.
        huge = struct.pack("<II6iiiiiqqqqqQiiqqqq", 0x5458564B, 2, lay.L, lay.H, lay.D, lay.E, lay.BS, lay.C,
                           NB, 0, lay.L, 0, 0, n, 1 << 62, nc, 0, 0, 0, 0, 0, 0, 0, 0)
        assert len(huge) == 136
        bad2 = _connect(sock)
        bad2.sendall(huge)
        bad2.close()
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        c = _connect(sock)
        kvx.kv_tier_load(c.fileno(), kvx.Cache(dB, lay.kv, NB), np.arange(lay.nblk(n), dtype=np.int32), n,
                         np.arange(nc), None)
        c.close()
        out, _ = p.communicate(timeout=90)
    assert p.returncode == 0, out[-2000:]
    results = [ln for ln in out.splitlines() if ln.startswith("TIER")][-1].split(" ", 1)[1].split(";")
    assert sorted(r == "ok" for r in results) == [False, False, True], results
    assert sum("malformed" in r for r in results) == 2, results


def _start_native_tier(sock, lay, slots, mode, nconn, dump, index_slots):
    return _start_tier(sock, lay, slots, mode, nconn, dump, role="tier-native", extra=(str(index_slots),))


def _finish_native(p):
    out, _ = p.communicate(timeout=90)
    assert p.returncode == 0, out[-2000:]
    assert [ln for ln in out.splitlines() if ln.startswith("TIER")][-1] == "TIER ok", out[-2000:]
    return out


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_prefix_store_and_external_hit(mode, tmp_path):
    """The tier as a prefix cache (library listener and threads, pool index): replica A stores a
    prompt; replica B asks for the same prompt and gets its whole chunks as an external hit
    (Sec. 3.1-3.2: hits are whole chunks), loaded bit-exactly; a prompt that diverges inside chunk
    3 hits 3 chunks; a new salt hits nothing; storing the prompt again writes nothing new."""
    lay = TINY
    n = 5 * lay.C + 100                      # 5 whole chunks and a partial one (not kept)
    NB = lay.nblk(n) + 9
    seed, salt = harness.sub_seed("prefix", mode), 11
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_native_tier(sock, lay, 8, mode, 3, dump, 8)
    with _serving(tier):
        r = subprocess.run([sys.executable, "-u", ROLES, "store-prefix", sock, *_dims(lay), str(NB), str(n), str(seed),
                            str(salt)], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0 and "STORED 5" in r.stdout, (r.stdout + r.stderr)[-3000:]
        tokens = harness.prompt_tokens(seed, n)
        btB = harness.block_table(seed + 2, NB, lay.nblk(n))
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        cB = kvx.Cache(dB, lay.kv, NB)
        torch.cuda.synchronize()
        c = _connect(sock)
        hit = kvx.kv_tier_load_prefix(c.fileno(), cB, btB, salt, tokens)
        got_B = dB.cpu()
        other = tokens.copy()
        other[3 * lay.C + 7] ^= 1
        assert kvx.kv_tier_load_prefix(c.fileno(), cB, btB, salt, other) == 3 * lay.C
        assert kvx.kv_tier_load_prefix(c.fileno(), cB, btB, salt + 1, tokens) == 0
        c.close()
        c2 = _connect(sock)                  # a third replica re-stores the same prompt: nothing new
        dC = torch.zeros_like(dB)
        torch.cuda.synchronize()
        assert kvx.kv_tier_store_prefix(c2.fileno(), kvx.Cache(dC, lay.kv, NB), btB, salt, tokens) == (0, 0)
        c2.close()
    out = _finish_native(tier)
    assert hit == 5 * lay.C
    A = host_cache(lay, NB, seed, "raw")
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    pool = np.load(dump)
    # The index gave chunks 0..4 slots 0..4 (lowest free first); slots 5..7 were never written.
    want_pool = oracle_pool(lay, A, btA, hit, np.arange(5), 8, POOL_SENT)
    assert np.array_equal(pool, want_pool), first_mismatch(pool, want_pool)
    want_B = oracle_unpack_into(lay, np.zeros_like(A), btB, hit, want_pool, np.arange(5))
    got = got_B.numpy().view(A.dtype).reshape(A.shape)
    assert np.array_equal(got, want_B), first_mismatch(got, want_B)
    assert "'entries': 5" in out and "'evictions': 0" in out


def _start_daemon(sock, lay, slots, mode, extra=()):
    from paper_2609_15021_amd import build
    assert os.path.exists(build.TIERD_BIN), "kvx_tierd not built; run __graft_entry__.build()"
    # The replicas here are torch processes: the daemon must run the HIP runtime torch ships, or
    # their IPC handles do not open in it.
    runtime = os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so")
    p = subprocess.Popen([build.TIERD_BIN, "--socket", sock, "--layout", ",".join(_dims(lay)), "--slots", str(slots),
                          "--mode", mode, "--staging-slots", "2", "--chunks-per-batch", "2", "--hip-runtime", runtime,
                          *extra],
                         stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    seen, t0 = [], time.time()
    while time.time() - t0 < 90:
        line = p.stdout.readline()
        if line.startswith("READY"):
            return p
        if not line and p.poll() is not None:
            break
        seen.append(line)
    p.kill()
    raise AssertionError(f"kvx_tierd did not start: {''.join(seen)[-2000:]}{p.stdout.read()[-2000:]}")


@pytest.mark.parametrize("mode", ["staged+zero_copy", "zero_copy"])
def test_tier_daemon_serves_a_prefix_cache(mode, tmp_path):
    """The standalone tier daemon (kvx_tierd: a native program over the C ABI) owns the pool and its
    index: replica A (a process) stores a prompt through it, replica B gets the whole-chunk hit; the
    pool the daemon dumps and B's cache equal the oracle's bytes."""
    lay = TINY
    n = 5 * lay.C + 100
    NB = lay.nblk(n) + 9
    seed, salt = harness.sub_seed("daemon", mode), 13
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.bin")
    d = _start_daemon(sock, lay, 8, mode, ("--index-slots", "8", "--connections", "2", "--fill", str(POOL_SENT),
                                           "--dump", dump))
    with _serving(d):
        r = subprocess.run([sys.executable, "-u", ROLES, "store-prefix", sock, *_dims(lay), str(NB), str(n), str(seed),
                            str(salt)], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0 and "STORED 5" in r.stdout, (r.stdout + r.stderr)[-3000:]
        tokens = harness.prompt_tokens(seed, n)
        btB = harness.block_table(seed + 2, NB, lay.nblk(n))
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        torch.cuda.synchronize()
        c = _connect(sock)
        hit = kvx.kv_tier_load_prefix(c.fileno(), kvx.Cache(dB, lay.kv, NB), btB, salt, tokens)
        got_B = dB.cpu()
        c.close()
        out, _ = d.communicate(timeout=90)
    assert d.returncode == 0 and "TIER ok" in out, out[-2000:]
    assert "entries=5 pending=0" in out, out[-2000:]
    assert hit == 5 * lay.C
    A = host_cache(lay, NB, seed, "raw")
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    pool = np.fromfile(dump, dtype=np.uint8)
    want_pool = oracle_pool(lay, A, btA, hit, np.arange(5), 8, POOL_SENT)
    assert np.array_equal(pool, want_pool), first_mismatch(pool, want_pool)
    want_B = oracle_unpack_into(lay, np.zeros_like(A), btB, hit, want_pool, np.arange(5))
    got = got_B.numpy().view(A.dtype).reshape(A.shape)
    assert np.array_equal(got, want_B), first_mismatch(got, want_B)


def test_tier_daemon_stops_cleanly_on_sigterm(tmp_path):
    """Serving without a connection limit, the daemon stops on SIGTERM: it stops accepting, reports
    the index and exits 0, removing its socket."""
    sock = str(tmp_path / "tier.sock")
    d = _start_daemon(sock, TINY, 4, "staged", ("--connections", "0"))
    c = _connect(sock)  # an idle replica connection that ends before the signal
    c.close()
    time.sleep(0.5)
    d.send_signal(signal.SIGTERM)
    try:
        out, _ = d.communicate(timeout=60)
    except subprocess.TimeoutExpired:
        d.kill()
        raise
    assert d.returncode == 0 and "TIER ok" in out and "STATS entries=0" in out, out[-2000:]
    assert not os.path.exists(sock)


def test_prefix_eviction_under_a_small_pool(tmp_path):
    """With 4 slots, storing a 3-chunk prompt and then a 3-chunk different prompt evicts the first
    prompt's tail (LRU, tails first): the first prompt then hits 1 chunk, the second all 3."""
    lay = TINY
    n = 3 * lay.C
    NB = lay.nblk(n) + 4
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_native_tier(sock, lay, 4, "staged", 3, dump, 4)
    with _serving(tier):
        for seed in (101, 202):
            r = subprocess.run([sys.executable, "-u", ROLES, "store-prefix", sock, *_dims(lay), str(NB), str(n),
                                str(seed), "5"], capture_output=True, text=True, timeout=120)
            assert r.returncode == 0 and "STORED 3" in r.stdout, (r.stdout + r.stderr)[-3000:]
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        cB = kvx.Cache(dB, lay.kv, NB)
        bt = np.arange(lay.nblk(n), dtype=np.int32)
        torch.cuda.synchronize()
        c = _connect(sock)
        assert kvx.kv_tier_load_prefix(c.fileno(), cB, bt, 5, harness.prompt_tokens(101, n)) == 1 * lay.C
        assert kvx.kv_tier_load_prefix(c.fileno(), cB, bt, 5, harness.prompt_tokens(202, n)) == 3 * lay.C
        c.close()
    out = _finish_native(tier)
    assert "'evictions': 2" in out


@pytest.mark.parametrize("mode", ["zero_copy", "staged", "staged+zero_copy"])
def test_hybrid_prefix_aligned_recovery_across_processes(mode, tmp_path):
    """The paper's hybrid case through the tier (Sec. 2.2): replica A stores a prompt's whole
    chunks plus the recurrent snapshot at its last whole-chunk boundary.  Replica B restores the
    prompt with aligned recovery: chunks and snapshot, bit-exact.  A prompt that diverges inside
    chunk 3 still shares 3 chunks of K/V pages but no snapshot at their boundary, so under aligned
    recovery it is no hit at all (attention pages alone do not recover the hybrid state), while an
    attention-only request hits the 3 chunks."""
    from tests.tier_roles import state_pages
    lay = TINY
    n = 5 * lay.C + 100
    NB = lay.nblk(n) + 9
    G, pb, npages, page_a, page_b = 3, 8192, 4, 2, 1
    seed, salt = harness.sub_seed("hybrid-tier", mode), 21
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_tier(sock, lay, 8, mode, 2, dump, role="tier-native", extra=("8", "2", str(G * pb)))
    with _serving(tier):
        r = subprocess.run([sys.executable, "-u", ROLES, "store-hybrid", sock, *_dims(lay), str(NB), str(n), str(seed),
                            str(salt), str(G), str(pb), str(npages), str(page_a)],
                           capture_output=True, text=True, timeout=120)
        assert r.returncode == 0 and "STORED 5 1" in r.stdout, (r.stdout + r.stderr)[-3000:]
        tokens = harness.prompt_tokens(seed, n)
        btB = harness.block_table(seed + 2, NB, lay.nblk(n))
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        dS = torch.zeros((G, npages, pb), dtype=torch.uint8, device=DEV)
        cB, sB = kvx.Cache(dB, lay.kv, NB), kvx.State(dS, pb, npages)
        torch.cuda.synchronize()
        c = _connect(sock)
        hit = kvx.kv_tier_load_prefix(c.fileno(), cB, btB, salt, tokens, state=sB, state_page=page_b)
        got_B, got_S = dB.cpu(), dS.cpu().numpy()
        other = tokens.copy()
        other[3 * lay.C + 7] ^= 1
        assert kvx.kv_tier_load_prefix(c.fileno(), cB, btB, salt, other, state=sB, state_page=page_b) == 0
        assert kvx.kv_tier_load_prefix(c.fileno(), cB, btB, salt, other) == 3 * lay.C
        c.close()
    _finish_native(tier)
    assert hit == 5 * lay.C
    A = host_cache(lay, NB, seed, "raw")
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    want_pool = oracle_pool(lay, A, btA, hit, np.arange(5), 8, POOL_SENT)
    want_B = oracle_unpack_into(lay, np.zeros_like(A), btB, hit, want_pool, np.arange(5))
    got = got_B.numpy().view(A.dtype).reshape(A.shape)
    assert np.array_equal(got, want_B), first_mismatch(got, want_B)
    pages_A = state_pages(seed, G, npages, pb)
    assert np.array_equal(got_S[:, page_b], pages_A[:, page_a])
    assert not got_S[:, [p for p in range(npages) if p != page_b]].any()


def test_two_replicas_store_at_the_same_time(tmp_path):
    """Two replica processes store different prompts through one tier concurrently (one native
    thread each, requests served one at a time); a third replica then hits both prompts whole."""
    lay = TINY
    n = 3 * lay.C
    NB = lay.nblk(n) + 4
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_tier(sock, lay, 8, "staged", 3, dump, role="tier-native", extra=("8",))
    with _serving(tier):
        procs = [subprocess.Popen([sys.executable, "-u", ROLES, "store-prefix", sock, *_dims(lay), str(NB), str(n),
                                   str(seed), "9"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
                 for seed in (303, 404)]
        outs = [p.communicate(timeout=120)[0] for p in procs]
        assert all(p.returncode == 0 and "STORED 3" in o for p, o in zip(procs, outs)), outs
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
        cB = kvx.Cache(dB, lay.kv, NB)
        bt = np.arange(lay.nblk(n), dtype=np.int32)
        torch.cuda.synchronize()
        c = _connect(sock)
        for seed in (303, 404):
            assert kvx.kv_tier_load_prefix(c.fileno(), cB, bt, 9, harness.prompt_tokens(seed, n)) == n
            got = dB.cpu().numpy().view(np.uint16)
            A = host_cache(lay, NB, seed, "raw")
            btA = harness.block_table(seed + 1, NB, lay.nblk(n))
            assert np.array_equal(got[:, bt], A[:, btA]), f"prompt {seed} restored wrong bytes"
        c.close()
    _finish_native(tier)


@pytest.mark.parametrize("i", range(6))
def test_random_layouts_through_the_tier(i, tmp_path):
    """Seeded layouts of the random-layout tests (head-major, packed blocks) stored by a replica
    process through the tier and restored by this process, each case in one of the three mode
    settings: the pool the tier dumps and the restored cache equal the oracle's bytes."""
    from tests.test_gpu_fuzz import _case
    lay, n, NB, _, _, _, _ = _case(7 * i + 3)
    mode = ["zero_copy", "staged", "staged+zero_copy"][i % 3]
    nc = lay.nc(n)
    seed = harness.sub_seed("tier-fuzz", i)
    print(f"[tier-fuzz] case {i} {mode}: L{lay.L} H{lay.H} D{lay.D} E{lay.E} BS{lay.BS} C{lay.C} n={n} NB={NB}",
          flush=True)
    sock, dump = str(tmp_path / "tier.sock"), str(tmp_path / "pool.npy")
    tier = _start_tier(sock, lay, nc + 1, mode, 2, dump)
    with _serving(tier):
        _store_process(sock, lay, NB, n, seed, 0)
        btB = harness.block_table(seed + 2, NB, lay.nblk(n))
        dB = torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=TORCH_INT[lay.E], device=DEV)
        s = torch.cuda.Stream()
        torch.cuda.synchronize()
        c = _connect(sock)
        kvx.kv_tier_load(c.fileno(), kvx.Cache(dB, lay.kv, NB), btB, n, np.arange(nc), s)
        got_B = dB.cpu()
        c.close()
    _finish_tier(tier)
    A = host_cache(lay, NB, seed, "raw")
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    want_pool = oracle_pool(lay, A, btA, n, np.arange(nc), nc + 1, POOL_SENT)
    pool = np.load(dump)
    assert np.array_equal(pool, want_pool), first_mismatch(pool, want_pool)
    want_B = oracle_unpack_into(lay, np.zeros_like(A), btB, n, want_pool, np.arange(nc))
    got = got_B.numpy().view(A.dtype).reshape(A.shape)
    assert np.array_equal(got, want_B), first_mismatch(got, want_B)
