"""The C ABI on the CPU: exported symbols, host-only entry points (bit-exact
against the reference's integer side) and argument validation that must fail
before anything reaches a GPU."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

from oracle import partition as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2608_01785_amd", "libhorizon.so")
HEADER = os.path.join(ROOT, "include", "horizon.h")


@pytest.fixture(scope="module")
def b():
    if not os.path.exists(LIB):
        pytest.skip("libhorizon.so not built")
    from paper_2608_01785_amd import binding
    binding.lib()
    return binding


def declared_functions():
    import re
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:hs_status|const char\*)\s+(hs_\w+)\(", text, re.M)))


def test_every_declared_symbol_is_exported(b):
    names = declared_functions()
    assert len(names) >= 14
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], stdout=subprocess.PIPE, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    assert set(b.SYMBOLS) == set(names)
    for n in names:
        getattr(b.lib(), n)


def test_status_strings(b):
    assert b.lib().hs_status_string(0) == b"HS_OK"
    assert b.lib().hs_status_string(3) == b"HS_ERR_BUDGET"


@pytest.mark.parametrize("c", [1, 7, 8, 63, 64, 96, 100, 128, 160, 192, 250, 256])
def test_partition_matches_reference_default_topology(b, c):
    t = b.hs_default_topology(256, 8)
    xcc, se, cu = P.default_topology()
    assert list(t.xcc) == xcc and list(t.se) == se and list(t.cu) == cu
    assert b.hs_cu_partition(t, c) == P.cu_partition(xcc, se, cu, 8, c)


def test_partition_matches_reference_random_topologies(b):
    rng = np.random.default_rng(0)
    for trial in range(20):
        n_xcc = int(rng.choice([1, 2, 4, 8]))
        per = int(rng.integers(4, 33))
        n = n_xcc * per
        xcc = rng.permutation(np.repeat(np.arange(n_xcc), per)).tolist()
        se = rng.integers(0, 4, size=n).tolist()
        cu = rng.integers(0, 16, size=n).tolist()
        t = b.topology_from_lists(xcc, se, cu, n_xcc)
        for c in rng.integers(1, n + 1, size=5).tolist() + [n]:
            assert b.hs_cu_partition(t, c) == P.cu_partition(xcc, se, cu, n_xcc, c), (trial, c)


@pytest.mark.parametrize("c", [0, -5, 257])
def test_partition_rejects_budget(b, c):
    t = b.hs_default_topology()
    with pytest.raises(b.HorizonError) as e:
        b.hs_cu_partition(t, c)
    assert e.value.status == b.HS_ERR_BUDGET


def test_plan_metadata_matches_reference(b):
    from paper_2608_01785_amd import workloads as W
    cases = [([0, 96, 224], None), ([0, 2, 2, 5], [3, 0, 7])]
    lengths, ctx = W.thinker_mixed_layout()
    off = np.concatenate([[0], np.cumsum(lengths)])
    cases.append((off.tolist(), ctx.tolist()))
    tb = W.thinker_batch(hidden=8)
    cases.append((tb.seq_offsets.tolist(), None))
    for off, ctx in cases:
        pos, sid = b.hs_plan_metadata(off, ctx)
        rpos, rsid = P.plan_metadata(off, ctx)
        np.testing.assert_array_equal(pos, rpos)
        np.testing.assert_array_equal(sid, rsid)
    for bad in ([1, 3], [0, 5, 4]):
        with pytest.raises(b.HorizonError) as e:
            b.hs_plan_metadata(bad)
        assert e.value.status == b.HS_ERR_INVALID_ARG


def test_workspace_size_monotone_and_validated(b):
    from paper_2608_01785_amd import workloads as W
    s1 = b.hs_workspace_size(W.THINKER, 1000, 4, 1000)
    s2 = b.hs_workspace_size(W.THINKER, 2000, 4, 1000)
    s3 = b.hs_workspace_size(W.THINKER, 2000, 8, 4000)
    assert 0 < s1 < s2 < s3
    import dataclasses
    bad = dataclasses.replace(W.THINKER, head_dim=96)
    with pytest.raises(b.HorizonError) as e:
        b.hs_workspace_size(bad, 10, 1, 10)
    assert e.value.status == b.HS_ERR_UNSUPPORTED
    bad = dataclasses.replace(W.THINKER, n_kv_heads=5)
    with pytest.raises(b.HorizonError) as e:
        b.hs_workspace_size(bad, 10, 1, 10)
    assert e.value.status == b.HS_ERR_INVALID_ARG


def _forward_null_ctx(b, cfg, offsets, ctx_lens=None, x_in=1 << 20, x_out=2 << 20, kv=None, n_layers=1):
    """Call the forward with a null context and fake (never dereferenced) pointers."""
    from paper_2608_01785_amd import binding
    w = (binding.LayerWeights * n_layers)()
    for i in range(n_layers):
        for name in ("ln1", "w_qkv", "w_o", "ln2", "w_gate_up", "w_down"):
            setattr(w[i], name, 0x1000)
    off = (ctypes.c_int32 * len(offsets))(*offsets)
    cl = None if ctx_lens is None else (ctypes.c_int32 * len(ctx_lens))(*ctx_lens)
    st = b.lib().hs_shared_stage_forward(None, ctypes.byref(binding.LayerCfg.of(cfg)), w, n_layers, x_in, x_out,
                                         off, cl, len(offsets) - 1, kv, 256, None, 0x3000, 1 << 30)
    return st, b.hs_last_error()


def test_forward_validation_fails_before_any_gpu_work(b):
    from paper_2608_01785_amd import workloads as W
    c = W.TINY
    st, msg = _forward_null_ctx(b, c, [0, 4, 9])
    assert st == b.HS_ERR_INVALID_ARG and "context" in msg
    st, msg = _forward_null_ctx(b, c, [0, 4, 3])
    assert st == b.HS_ERR_INVALID_ARG and "decrease" in msg
    st, msg = _forward_null_ctx(b, c, [1, 4])
    assert st == b.HS_ERR_INVALID_ARG
    st, msg = _forward_null_ctx(b, c, [0, 4], x_in=5, x_out=5)
    assert st == b.HS_ERR_INVALID_ARG and "alias" in msg
    st, msg = _forward_null_ctx(b, c, [0, 4], ctx_lens=[3])
    assert st == b.HS_ERR_INVALID_ARG and "cache" in msg
    st, msg = _forward_null_ctx(b, c, [0, 4], ctx_lens=[-1])
    assert st == b.HS_ERR_INVALID_ARG
    import dataclasses
    st, msg = _forward_null_ctx(b, dataclasses.replace(c, hidden=320), [0, 4])
    assert st == b.HS_ERR_UNSUPPORTED


def test_extents_beyond_32_bit_byte_offsets_are_rejected(b):
    # The GEMMs' buffer resources count bytes in 32 bits: at FFN 18944 the
    # SwiGLU output of 113,360 rows takes 2^32 bytes or more.  Such a batch
    # must fail before any GPU work instead of reading zeros past the end.
    from paper_2608_01785_amd import workloads as W
    c = W.THINKER
    assert 113360 * c.ffn * 2 >= 1 << 32 > 113359 * c.ffn * 2
    st, msg = _forward_null_ctx(b, c, [0, 113360])
    assert st == b.HS_ERR_UNSUPPORTED and "SwiGLU" in msg, msg
    st, msg = _forward_null_ctx(b, c, [0, 60000, 113360])
    assert st == b.HS_ERR_UNSUPPORTED, msg
    st, msg = _forward_null_ctx(b, c, [0, 113359])
    assert st == b.HS_ERR_INVALID_ARG and "context" in msg, msg           # every check passed
    # A weight matrix of 2^32 bytes or more.
    import dataclasses
    big = dataclasses.replace(c, hidden=8192, ffn=131072)
    st, msg = _forward_null_ctx(b, big, [0, 4])
    assert st == b.HS_ERR_UNSUPPORTED and "w_gate_up" in msg, msg
    # A cache page that single-row attention cannot address.
    kv = _fake_kv(b, 1, 1 << 23)
    st, msg = _forward_null_ctx(b, c, [0, 4], ctx_lens=[0], kv=ctypes.byref(kv))
    assert st == b.HS_ERR_UNSUPPORTED and "page" in msg, msg
    kv = _fake_kv(b, 1, 1 << 22)
    st, msg = _forward_null_ctx(b, c, [0, 4], ctx_lens=[0], kv=ctypes.byref(kv))
    assert st == b.HS_ERR_INVALID_ARG and "context" in msg, msg


def _fake_kv(b, n_slots, page, table=None, n_layers=1):
    """A cache struct with fake (never dereferenced) layer pointers and an optional block table."""
    from paper_2608_01785_amd import binding
    return binding._kv_struct(([0x5000] * n_layers, [0x6000] * n_layers, n_slots, page, table))


def test_paged_cache_validation_fails_before_any_gpu_work(b):
    from paper_2608_01785_amd import workloads as W
    c = W.TINY

    def call(offsets, ctx_lens, n_slots, page, table):
        kv = _fake_kv(b, n_slots, page, None if table is None else np.asarray(table, np.int32))
        return _forward_null_ctx(b, c, offsets, ctx_lens=ctx_lens, kv=ctypes.byref(kv))

    # Valid: two sequences share a read-only prefix page (slot 3) and write their own pages.
    st, msg = call([0, 10, 30], [128, 200], 6, 128, [[3, 0, 5], [3, 1, 5]])
    assert st == b.HS_ERR_INVALID_ARG and "context" in msg, msg
    # The same batch without a table needs positions < max_ctx.
    st, msg = call([0, 10, 30], [128, 200], 6, 128, None)
    assert st == b.HS_ERR_INVALID_ARG and "exceeds max_ctx" in msg, msg
    # Page size not a multiple of 64.
    st, msg = call([0, 10], [0], 6, 96, [[0]])
    assert st == b.HS_ERR_INVALID_ARG and "multiple of 64" in msg, msg
    # Slot index outside the pool.
    st, msg = call([0, 10], [100], 2, 64, [[0, 2]])
    assert st == b.HS_ERR_INVALID_ARG and "outside" in msg, msg
    # Positions beyond the sequence's pages.
    st, msg = call([0, 10], [120], 6, 64, [[0, 1]])
    assert st == b.HS_ERR_INVALID_ARG and "beyond" in msg, msg
    # One sequence listing a slot twice.
    st, msg = call([0, 10], [120], 6, 64, [[4, 4, 1]])
    assert st == b.HS_ERR_INVALID_ARG and "twice" in msg, msg
    # A page receiving rows of one sequence and reached by another.
    st, msg = call([0, 10, 11], [60, 70], 6, 64, [[0, 1], [0, 1]])
    assert st == b.HS_ERR_INVALID_ARG and "other sequences" in msg, msg
    # Entries past the pages a sequence reaches are not read (-1 there is fine).
    st, msg = call([0, 10], [0], 6, 64, [[2, -1, -1]])
    assert st == b.HS_ERR_INVALID_ARG and "context" in msg, msg


def test_mrope_validation_fails_before_any_gpu_work(b):
    import dataclasses
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd import workloads as W

    def call(cfg, offsets, pos3):
        w = (binding.LayerWeights * 1)()
        for name in ("ln1", "w_qkv", "w_o", "ln2", "w_gate_up", "w_down"):
            setattr(w[0], name, 0x1000)
        off = (ctypes.c_int32 * len(offsets))(*offsets)
        p = None if pos3 is None else np.ascontiguousarray(pos3, np.int32)
        st = b.lib().hs_shared_stage_forward_mrope(
            None, ctypes.byref(binding.LayerCfg.of(cfg)), w, 1, 1 << 20, 2 << 20, off, None, len(offsets) - 1, None,
            None if p is None else p.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 256, None, 0x3000, 1 << 30)
        return st, b.hs_last_error()

    c = dataclasses.replace(W.TINY, mrope_sections=(8, 12, 12))
    good = W.mrope_positions([10, 6], [4, 0])
    st, msg = call(c, [0, 10, 16], good)
    assert st == b.HS_ERR_INVALID_ARG and "context" in msg, msg          # every check passed
    st, msg = call(c, [0, 10, 16], None)
    assert st == b.HS_ERR_INVALID_ARG and "positions3" in msg, msg
    st, msg = call(W.TINY, [0, 10, 16], good)
    assert st == b.HS_ERR_INVALID_ARG and "mrope_sections" in msg, msg
    bad = good.copy()
    bad[1, 3] = 10                                                       # the largest row position is 9
    st, msg = call(c, [0, 10, 16], bad)
    assert st == b.HS_ERR_INVALID_ARG and "outside" in msg, msg
    for sec in ((8, 12, 8), (6, 14, 12), (-4, 24, 12)):
        st, msg = call(dataclasses.replace(W.TINY, mrope_sections=sec), [0, 10, 16], good)
        assert st == b.HS_ERR_INVALID_ARG and "multiples of 4" in msg, msg


def test_paged_workspace_size(b):
    from paper_2608_01785_amd import workloads as W
    c = W.TALKER
    plain = b.hs_workspace_size(c, 128, 128, 4096)
    assert b.hs_workspace_size_paged(c, 128, 128, 4096, 0) == plain
    assert b.hs_workspace_size_paged(c, 128, 128, 4096, 1024) >= plain
    # Smaller pages cut single-row attention into more work units.
    assert b.hs_workspace_size_paged(c, 128, 128, 4096, 64) > b.hs_workspace_size_paged(c, 128, 128, 4096, 1024)
    for bad in (-64, 100):
        with pytest.raises(b.HorizonError) as e:
            b.hs_workspace_size_paged(c, 128, 128, 4096, bad)
        assert e.value.status == b.HS_ERR_INVALID_ARG


def test_host_planner_under_sanitizers(tmp_path):
    """Build the host-only planner, controller and temporal scheduler with g++ and ASan/UBSan and drive them."""
    gxx = "g++"
    drv = tmp_path / "drv.cpp"
    drv.write_text(r'''
#include "horizon.h"
#include "plan.h"
#include "decode_policy.h"
#include <stdio.h>
#include <vector>
// A paged plan: every row's key/value offset and every single-row unit's page
// base follow the block table, and every unit's keys stay inside its page.
static int paged_plan_check() {
  hs_layer_cfg c = {256, 4, 2, 64, 1024, 1e-6f, 1e4f};
  const int P = 64, pps = 40, n_slots = 200, dh = 64, hkv = 2;
  int off[] = {0, 1, 2, 150, 151};
  int ctx[] = {0, 1999, 100, 64};
  std::vector<int> table(4 * pps, -1);
  int next = 0;
  for (int b = 0; b < 4; ++b) {
    const int end = ctx[b] + off[b + 1] - off[b];
    for (int j = 0; j * P < end; ++j) table[b * pps + j] = (next++ * 7) % n_slots;
  }
  if (hs::check_block_table(table.data(), pps, n_slots, P, off, ctx, 4) != HS_OK) return 1;
  hs::KvPlacement kv;
  kv.cache = true; kv.max_ctx = P; kv.table = table.data(); kv.pages_per_seq = pps;
  hs::Plan plan;
  if (hs::build_plan(c, off, ctx, 4, kv, &plan) != HS_OK) return 2;
  const int64_t slot = int64_t(hkv) * P * dh;
  const int64_t* koff = reinterpret_cast<const int64_t*>(plan.image.data() + plan.k_off);
  const int64_t* voff = reinterpret_cast<const int64_t*>(plan.image.data() + plan.v_off);
  for (int b = 0; b < 4; ++b)
    for (int t = off[b]; t < off[b + 1]; ++t) {
      const int p = ctx[b] + t - off[b], s = table[b * pps + p / P], i = p % P;
      if (koff[t] != s * slot + int64_t(i) * dh) return 3;
      if (voff[t] != s * slot + int64_t(i / 32) * 32 * dh + i % 32) return 4;
    }
  if (plan.unit_keys != 64 || plan.page_keys != P) return 5;
  for (int it = 0; it < plan.n_dec_items; ++it) {
    const int32_t* r = reinterpret_cast<const int32_t*>(plan.image.data() + plan.dec_items + size_t(it) * 32);
    const int64_t base = *reinterpret_cast<const int64_t*>(plan.image.data() + plan.dec_items + size_t(it) * 32 + 16);
    int b = 0;
    while (off[b] != r[0]) ++b;
    const int k_begin = r[2] * plan.unit_keys;
    if (k_begin >= r[1] || base != table[b * pps + k_begin / P] * slot) return 6;
    if (k_begin % P + plan.unit_keys > P) return 7;  // the unit stays in its page
  }
  if (hs::dec_unit_keys(128, 1024) != 512 || hs::dec_unit_keys(64, 192) != 64 || hs::dec_unit_keys(64, 0) != 1024)
    return 8;
  return 0;
}
int main() {
  hs_topology t;
  if (hs_default_topology(256, 8, &t) != HS_OK) return 1;
  uint32_t s[8], d[8];
  for (int c = 1; c <= 256; ++c) if (hs_cu_partition(&t, c, s, d) != HS_OK) return 2;
  if (hs_cu_partition(&t, 0, s, d) != HS_ERR_BUDGET) return 3;
  int off[] = {0, 3, 3, 10}; int ctx[] = {5, 0, 2};
  std::vector<int> pos(10), sid(10);
  if (hs_plan_metadata(off, ctx, 3, pos.data(), sid.data()) != HS_OK) return 4;
  if (pos[9] != 8 || sid[9] != 2) return 5;
  hs_layer_cfg c = {3584, 28, 4, 128, 18944, 1e-6f, 1e4f};
  size_t n = 0;
  if (hs_workspace_size(&c, 10515, 8, 2048, &n) != HS_OK || n == 0) return 6;
  size_t np = 0;
  if (hs_workspace_size_paged(&c, 10515, 8, 2048, 64, &np) != HS_OK || np < n) return 10;
  int ladder[] = {64, 96, 128, 160, 192};
  hs_controller_cfg cc = {256, 256, ladder, 5, 0.4, 0.8, 1};
  hs_controller* ctrl = nullptr;
  if (hs_controller_create(&cc, &ctrl) != HS_OK) return 7;
  hs_split sp;
  for (int i = 0; i < 1000; ++i)
    if (hs_controller_step(ctrl, i % 7 != 0, (i % 13) / 10.0, &sp) != HS_OK || sp.shared_cus + sp.down_cus != 256)
      return 8;
  hs_controller_destroy(ctrl);
  cc.n_ladder = 0;
  if (hs_controller_create(&cc, &ctrl) != HS_ERR_INVALID_ARG) return 9;
  if (paged_plan_check() != 0) return 11;
  hs_temporal_cfg tc = {2, 8, 2, 1.0, 3};
  hs_temporal* ts = nullptr;
  if (hs_temporal_create(&tc, &ts) != HS_OK) return 12;
  std::vector<hs_request_view> rq(40);
  std::vector<uint8_t> vis(40);
  hs_temporal_step_info ti;
  for (int k = 0; k < 500; ++k) {
    for (int i = 0; i < 40; ++i) rq[i] = {i % 2, (i % 7) == 0, double(i % 11) + 0.25 * k, 1.0 + (i % 3)};
    if (hs_temporal_step(ts, 0.5 * k, rq.data(), 40 - k % 40, vis.data(), &ti) != HS_OK || ti.step != k) return 13;
  }
  rq[0].remaining = 0.0;
  if (hs_temporal_step(ts, 0.0, rq.data(), 1, vis.data(), &ti) != HS_ERR_INVALID_ARG) return 14;
  hs_temporal_destroy(ts);
  printf("ok %zu\n", n);
  return 0;
}
''')
    exe = tmp_path / "drv"
    srcs = [os.path.join(ROOT, "paper_2608_01785_amd", "csrc", f) for f in ("plan.cpp", "controller.cpp", "temporal.cpp")]
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{os.path.join(ROOT, 'paper_2608_01785_amd', 'csrc')}",
           str(drv), *srcs, "-o", str(exe), "-ldl"]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    r = subprocess.run([str(exe)], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout


def test_binding_rejects_positions3_of_the_wrong_length(b):
    # The library reads 3 * T positions (T = the last offset); a shorter array
    # would be read past its end on the host, so the binding refuses it before
    # the call (no context or device memory is touched).
    import dataclasses
    from paper_2608_01785_amd import workloads as W
    c = dataclasses.replace(W.TINY, mrope_sections=(8, 12, 12))
    w = [{n: 0x1000 for n in ("ln1", "w_qkv", "w_o", "ln2", "w_gate_up", "w_down")}]
    short = W.mrope_positions([10, 5], [4, 0])                  # T = 15, offsets say 16
    with pytest.raises(ValueError, match="positions3"):
        b.hs_shared_stage_forward_mrope(None, c, w, 1 << 20, 2 << 20, [0, 10, 16], short, workspace=0x3000,
                                        ws_bytes=1 << 30)
    with pytest.raises(ValueError, match="positions3"):
        b.hs_downstream_decode_step_mrope(None, c, w, 1 << 20, 2 << 20, ([0x5000], [0x6000], 4, 64), [3, 4, 5],
                                          np.zeros((3, 2), np.int32), 128, workspace=0x3000, ws_bytes=1 << 30)
