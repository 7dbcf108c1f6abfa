"""Host-side checks of the C ABI library: it loads without a GPU and exports every declared symbol."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "canon.h")).read()
    return sorted(set(re.findall(r"\b(canon_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    import paper_2609_17380_amd.canon as C
    lib = C.lib()
    names = declared_symbols()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert C.version() == 1
    assert lib.canon_status_str(-4) == b"workspace too small"


def test_workspace_queries_without_gpu():
    import numpy as np
    import paper_2609_17380_amd.canon as C
    cfg = C.ModelCfg(16, 2048, 16, 128, 8192, 50304, 2048, 4, np.float32(1e-5))
    plan = C.DPPlan(1, 8, 1)
    ws = C.step_workspace_bytes(cfg, plan)
    assert 30e9 < ws < 80e9  # fits one MI355X next to the parameters and moments
    assert C.block_workspace_bytes(cfg, 1) > 0
    bad = C.ModelCfg(16, 2048, 15, 128, 8192, 50304, 2048, 4, np.float32(1e-5))  # heads * head_dim != d
    assert C.step_workspace_bytes(bad, plan) == 0


def test_oracle_and_library_share_no_source():
    lib_src = open(os.path.join(ROOT, "paper_2609_17380_amd", "csrc", "canon_dev.h")).read()
    orc = open(os.path.join(ROOT, "oracle", "canon_ref.c")).read()
    assert "canon_dev.h" not in orc and "canon.h" not in orc.replace("canon_ref.h", "")
    assert "canon_ref" not in lib_src


def test_host_validation_rejects_before_any_launch():
    # argument checks run on the host and return before anything is enqueued, so they need no GPU; the
    # pointers below are never dereferenced
    import ctypes
    import paper_2609_17380_amd.canon as C
    lib = C.lib()
    order = ctypes.byref(C.ORDER_V1)
    base = 1 << 32
    rows, cols = 64, 128
    n = rows * cols * 4
    x, dy, dx, rstd, gain, dg = base, base + n, base + 2 * n, base + 3 * n, base + 3 * n + 4096, base + 3 * n + 8192
    # dx overlapping dy, x, rstd or dgain is rejected (dx holds scratch before its values)
    for bad_dx in (dy + 4, x, rstd - 8, dg - 16):
        assert lib.canon_rownorm(order, C.BWD, rows, cols, x, gain, 1e-5, None, rstd, dy, bad_dx, dg, None) == C.EINVAL
    # a wrong order descriptor and a bad direction
    bad = C.Order(1, 31, 0, 1)
    assert lib.canon_rownorm(ctypes.byref(bad), C.FWD, rows, cols, x, gain, 1e-5, dx, rstd, None, None, None,
                             None) != C.OK
    assert lib.canon_rownorm(order, 7, rows, cols, x, gain, 1e-5, dx, rstd, None, None, None, None) == C.EINVAL
    # GEMM with negative sizes, softmax with rows not a multiple of cols
    assert lib.canon_gemm(order, 0, 0, -1, 4, 4, x, 4, dy, 4, dx, 4, None, None) == C.EINVAL
    # an unknown GEMM epilogue kind
    bad_epi = C.GemmEpilogue(7, 1.0)
    assert lib.canon_gemm(order, 0, 0, 4, 4, 4, x, 4, dy, 4, dx, 4, ctypes.byref(bad_epi), None) == C.EINVAL
    assert lib.canon_softmax_xent(order, C.SOFTMAX_CAUSAL, 10, 4, x, 1.0, 0, None, 1.0, 0.0, dx, None, None,
                                  None) == C.EINVAL
    # a negative window or z-loss weight
    assert lib.canon_softmax_xent(order, C.SOFTMAX_CAUSAL, 8, 4, x, 1.0, -1, None, 1.0, 0.0, dx, None, None,
                                  None) == C.EINVAL
    assert lib.canon_softmax_xent(order, C.XENT, 8, 4, x, 1.0, 0, x, 1.0, -1.0, dx, dy, None, None) == C.EINVAL
    # model configs: kv heads that do not divide the query heads, a bad flag, a negative window
    for fields in ({"n_kv_heads": 3}, {"qk_norm": 2}, {"swa_window": -1}, {"z_loss": -1.0}):
        cfg = C.ModelCfg(1, 64, 4, 16, 96, 97, 48, 1, 1e-5)
        for k_, v_ in fields.items():
            setattr(cfg, k_, v_)
        assert lib.canon_block_workspace_bytes(ctypes.byref(cfg), 1) == 0, fields
    # a step index below 1
    cfg = C.ModelCfg(1, 64, 4, 16, 96, 97, 48, 1, 1e-5)
    plan = C.DPPlan(1, 1, 1)
    ptrs = (ctypes.c_void_p * 9)(*([base] * 9))
    consts = C.AdamWConsts(*([0.1] * 9))
    for t in (0, -3):
        assert lib.canon_step(order, ctypes.byref(cfg), ctypes.byref(plan), ptrs, ptrs, ptrs, t, x, x, x,
                              ctypes.byref(consts), None, x, 1 << 30, x, None, None, None) == C.EINVAL
    # a per-step digest with a workspace off 256-byte alignment
    assert lib.canon_step(order, ctypes.byref(cfg), ctypes.byref(plan), ptrs, ptrs, ptrs, 1, x, x, x,
                          ctypes.byref(consts), None, x + 16, 1 << 40, x, None, x, None) == C.EINVAL
    # embedding backward: negative sizes, a missing pointer, too many positions, a small workspace
    assert lib.canon_embed_bwd(order, -1, 10, 4, x, dx, dy, x, 1 << 20, None) == C.EINVAL
    assert lib.canon_embed_bwd(order, 8, 10, 4, None, dx, dy, x, 1 << 20, None) == C.EINVAL
    assert lib.canon_embed_bwd(order, 1 << 25, 10, 4, x, dx, dy, x, 1 << 40, None) == C.EUNSUPPORTED
    assert lib.canon_embed_bwd(order, 8, 10, 4, x, dx, dy, x, 16, None) == C.EWORKSPACE
    # the allocation-free LSQ gradient beyond its array
    big = lib.canon_lsq_step_grad_noalloc_max_terms() // 8 + 1
    assert lib.canon_lsq_step_grad_noalloc(order, big, 8, x, dx, dy, rstd, None) == C.EUNSUPPORTED


def test_sha256_constants_in_the_device_source():
    # the round constants and initial state are the first 32 fraction bits of the cube roots of the first 64
    # primes and of the square roots of the first 8 (FIPS 180-4); integer roots keep this exact
    import re
    src = open(os.path.join(ROOT, "paper_2609_17380_amd", "csrc", "hash.hip")).read()
    k = [int(x, 16) for x in re.findall(r"0x([0-9a-f]{8})u", src[src.index("kSha256K"):src.index("kSha256H0")])]
    h0 = [int(x, 16) for x in re.findall(r"0x([0-9a-f]{8})u", src[src.index("kSha256H0"):src.index("rotr")])]
    primes = [p for p in range(2, 400) if all(p % q for q in range(2, int(p ** 0.5) + 1))][:64]

    def iroot(n, r):
        x = int(round(n ** (1.0 / r)))
        while x ** r > n:
            x -= 1
        while (x + 1) ** r <= n:
            x += 1
        return x

    assert k == [iroot(p << 96, 3) & 0xFFFFFFFF for p in primes]
    assert h0 == [iroot(p << 64, 2) & 0xFFFFFFFF for p in primes[:8]]


def _plan_record_shape(plan, next_):
    """What the plan record must hold after next_ pushes: the shard sum's presence and the stack levels."""
    accum, shard, rep = plan
    r = next_ // accum
    groups = r // shard
    return (r % shard) != 0, [L for L in range(30, -1, -1) if (groups >> L) & 1]


def test_plan_cursor_walk_without_gpu():
    """With n = 0 the plan calls launch nothing, so the host record's whole walk (position, shard sum, the
    binary-carry stack of Algorithm 2, slot use) can be followed on the CPU, including persisting the record
    and resuming from its bytes after every push."""
    import paper_2609_17380_amd.canon as C
    STATE = 1 << 20  # a stand-in address: with n = 0 nothing reads or writes it
    for plan in [(1, 8, 1), (2, 4, 1), (1, 2, 4), (3, 1, 5), (2, 3, 3), (1, 1, 13), (1, 1, 64), (2, 1, 100)]:
        p = C.DPPlan(*plan)
        nslots = (1 if plan[0] > 1 else 0) + int(plan[2]).bit_length() + 1
        assert C.plan_state_bytes(p, 0) == 0
        assert C.plan_state_bytes(p, 100) == 4 * 128 * nslots  # slots of 64-float multiples
        total = plan[0] * plan[1] * plan[2]
        cur = C.plan_begin(p, 0)
        for i in range(total):
            C.plan_push(cur, None, STATE, state_bytes=0, stream=0)
            cur = C.PlanCursor.from_buffer_copy(bytes(cur))  # persisted and resumed
            has_inner, levels = _plan_record_shape(plan, i + 1)
            assert cur.next == i + 1
            assert (cur.inner >= 0) == has_inner
            assert list(cur.level[:cur.depth]) == levels
            used = list(cur.slot[:cur.depth]) + ([cur.inner] if has_inner else [])
            assert len(set(used)) == len(used) and all(0 <= s < nslots for s in used)
        assert cur.depth == bin(plan[2]).count("1")
        C.plan_finish(cur, STATE, None, state_bytes=0, stream=0)


def test_plan_cursor_validation_without_gpu():
    """Records the calls cannot produce are rejected before any launch, and the record is left unchanged."""
    import paper_2609_17380_amd.canon as C
    p = C.DPPlan(1, 1, 6)
    n = 1000
    need = C.plan_state_bytes(p, n)
    STATE, GRAD = 1 << 20, 1 << 21  # never dereferenced: every case below fails validation first
    cur = C.plan_begin(p, 0)
    for _ in range(3):  # three replicas in: levels 1 and 0
        C.plan_push(cur, None, STATE, state_bytes=0, stream=0)
    good = bytes(cur)
    good_n = C.PlanCursor.from_buffer_copy(good)
    good_n.n = n

    def mutated(fn):
        c = C.PlanCursor.from_buffer_copy(bytes(good_n))
        fn(c)
        return c

    bad = [
        mutated(lambda c: setattr(c, "next", 7)),                        # beyond the plan's 6 microbatches
        mutated(lambda c: setattr(c, "next", -1)),
        mutated(lambda c: setattr(c, "depth", 1)),                       # stack shape not that of 3 replicas
        mutated(lambda c: c.level.__setitem__(0, 0)),
        mutated(lambda c: c.slot.__setitem__(1, c.slot[0])),             # one slot twice
        mutated(lambda c: c.slot.__setitem__(0, 9)),                     # slot out of range
        mutated(lambda c: setattr(c, "inner", 2)),                       # a shard sum with dp_shard = 1
        mutated(lambda c: setattr(c, "plan", C.DPPlan(0, 1, 6))),
        mutated(lambda c: setattr(c, "n", -5)),
    ]
    for c in bad:
        before = bytes(c)
        for call in (lambda: C.plan_push(c, GRAD, STATE, state_bytes=need, stream=0),
                     lambda: C.plan_finish(c, STATE, GRAD, state_bytes=need, stream=0)):
            try:
                call()
                raise AssertionError("accepted a record the calls cannot produce")
            except C.CanonError as e:
                assert e.status == C.EINVAL, e
            assert bytes(c) == before
    # a valid record: a misaligned or too small state, a missing gradient
    for kw, args in [(dict(state_bytes=need), (GRAD, STATE + 4)), (dict(state_bytes=need - 4), (GRAD, STATE)),
                     (dict(state_bytes=need), (None, STATE))]:
        c = C.PlanCursor.from_buffer_copy(bytes(good_n))
        try:
            C.plan_push(c, *args, stream=0, **kw)
            raise AssertionError("accepted")
        except C.CanonError as e:
            assert e.status in (C.EINVAL, C.EWORKSPACE)
        assert bytes(c) == bytes(good_n)
    # finish before the last push
    try:
        C.plan_finish(C.PlanCursor.from_buffer_copy(bytes(good_n)), STATE, GRAD, state_bytes=need, stream=0)
        raise AssertionError("accepted")
    except C.CanonError as e:
        assert e.status == C.EINVAL
