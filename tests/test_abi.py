"""The C ABI without a GPU: the library loads, exports every function that
include/cascade.h declares, the ctypes mirror has the header's exact struct
layout, and host-side argument checks return their codes before any launch."""
import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2608_06557_amd import cascade

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cascade.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(cascade.LIB_PATH):
        from paper_2608_06557_amd import build
        build.build()
    return cascade.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(cascade_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(cascade.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", cascade.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (\w+)$", out, flags=re.M))
    for n in names:
        assert n in exported, n
        assert hasattr(lib, n)


STRUCTS = {
    "cascade_requests_t": cascade.Requests, "cascade_block_table_t": cascade.BlockTable,
    "cascade_tier_state_t": cascade.TierState, "cascade_params_t": cascade.Params,
    "cascade_move_t": cascade.Move, "cascade_outputs_t": cascade.Outputs,
    "cascade_kv_pool_t": cascade.KvPool, "cascade_tier_table_t": cascade.TierTable,
    "cascade_tier_chain_t": cascade.TierChain,
}


def test_demotion_record_layout_matches_header(tmp_path):
    dt = cascade.DEMOTION_DTYPE
    src = tmp_path / "dem.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "cascade.h"\n'
                   'int main(){printf("%zu %zu %zu %zu %zu\\n", sizeof(cascade_demotion_t),'
                   'offsetof(cascade_demotion_t, hash), offsetof(cascade_demotion_t, last_use_ns),'
                   'offsetof(cascade_demotion_t, src_slot), offsetof(cascade_demotion_t, pad));'
                   'return 0;}')
    exe = tmp_path / "dem"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], check=True, capture_output=True,
                                          text=True).stdout.split()]
    assert got == [dt.itemsize] + [dt.fields[f][1] for f in ("hash", "last_use_ns", "src_slot",
                                                              "pad")]


def test_struct_layout_matches_header(tmp_path):
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "cascade.h"', "int main(){"]
    for cname, py in STRUCTS.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines.append("return 0;}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    got = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    seen = 0
    for line in got:
        if not line:
            continue
        cname, field, val = line.split()
        py = STRUCTS[cname]
        if field == "size":
            assert C.sizeof(py) == int(val), cname
        else:
            assert getattr(py, field).offset == int(val), (cname, field)
        seen += 1
    assert seen == sum(len(p._fields_) + 1 for p in STRUCTS.values())


def test_constants_match_header():
    text = open(HEADER).read()
    defs = dict((k, int(v)) for k, v in
                re.findall(r"#define CASCADE_(\w+)\s+\(?(-?\d+)\)?", text))
    for k, v in defs.items():
        name = k[5:] if k.startswith("INFO_") and k != "INFO_LEN" else k
        if k == "INFO_LEN":
            assert cascade.INFO_LEN == v
        elif k.startswith("INFO_"):
            assert getattr(cascade, k) == v, k
        else:
            assert getattr(cascade, name) == v, k


def test_workspace_size(lib):
    prev = 0
    for n in [0, 1, 1000, 65536, 262144, 1 << 20]:
        b = cascade.cascade_step_workspace_bytes(n)
        assert b % 256 == 0 and b >= prev
        prev = b
    assert cascade.cascade_step_workspace_bytes(-1) == 0
    assert cascade.cascade_step_workspace_bytes((1 << 20) + 1) == 0


def _valid_args():
    import paper_2608_06557_amd.synth as synth
    p = cascade.make_params(synth.make_params(0))
    fake = 4096  # never dereferenced: every case below fails a host-side check
    req = cascade.Requests(4, *([fake] * 10))
    table = cascade.BlockTable(fake, fake)
    tier = cascade.TierState(100, 10, fake)
    out = cascade.Outputs(*([fake] * 12), 10, 10, 10, fake)
    return req, table, tier, p, out


def test_host_checks_return_einval_without_launch(lib):
    req, table, tier, p, out = _valid_args()
    ws = cascade.cascade_step_workspace_bytes(4)
    f = lambda **kw: cascade.cascade_step(kw.get("req", req), kw.get("table", table),
                                          kw.get("tier", tier), kw.get("p", p),
                                          kw.get("out", out), kw.get("ws", 1 << 20),
                                          kw.get("wsb", ws), 0)
    assert lib.cascade_step(None, None, None, None, None, None, 0, None) == cascade.EINVAL
    bad = cascade.Params.from_buffer_copy(p)
    bad.gamma_q16 = 1000
    assert f(p=bad) == cascade.EINVAL
    bad = cascade.Params.from_buffer_copy(p)
    bad.num_classes = 0
    assert f(p=bad) == cascade.EINVAL
    r2 = cascade.Requests.from_buffer_copy(req)
    r2.n = -1
    assert f(req=r2) == cascade.EINVAL
    r2.n = (1 << 20) + 1
    assert f(req=r2) == cascade.EINVAL
    r2 = cascade.Requests.from_buffer_copy(req)
    r2.n_in = None
    assert f(req=r2) == cascade.EINVAL
    t2 = cascade.TierState(100, 101, 4096)
    assert f(tier=t2) == cascade.EINVAL
    o2 = cascade.Outputs.from_buffer_copy(out)
    o2.pack_capacity = -1
    assert f(out=o2) == cascade.EINVAL
    o2 = cascade.Outputs.from_buffer_copy(out)
    o2.unpack_hazard = 4096                           # one hazard array without the other
    assert f(out=o2) == cascade.EINVAL
    assert f(ws=(1 << 20) + 8) == cascade.EINVAL       # workspace not 256-byte aligned
    assert f(wsb=ws - 1) == cascade.ENOSPC


def test_copy_host_checks(lib):
    pool = cascade.KvPool(4096, 32, 10, 32768, 65536, 32768, 32768)
    n = C.c_int32(1)
    ok = dict(pool=pool, staging=4096, staging_slots=4, moves=4096,
              n_moves_dev=C.addressof(n), max_moves=4, status_dev=0, stream=0)

    def call(fn, **kw):
        a = dict(ok)
        a.update(kw)
        return fn(a["pool"], a["staging"], a["staging_slots"], a["moves"], a["n_moves_dev"],
                  a["max_moves"], a["status_dev"], a["stream"])
    for fn in (cascade.cascade_pack, cascade.cascade_unpack):
        assert call(fn, staging=0) == cascade.EINVAL
        assert call(fn, staging=4100) == cascade.EINVAL            # misaligned
        assert call(fn, max_moves=-1) == cascade.EINVAL
        assert call(fn, pool=cascade.KvPool(4096, 0, 10, 32768, 0, 0, 0)) == cascade.EINVAL
        assert call(fn, pool=cascade.KvPool(4096, 2, 10, 24, 0, 0, 0)) == cascade.EINVAL
        assert call(fn, pool=cascade.KvPool(4096, 2, 10, 32, 8, 0, 0)) == cascade.EINVAL
        assert call(fn, max_moves=0) == cascade.OK                   # nothing to launch


def test_fused_copy_host_checks(lib):
    pool = cascade.KvPool(4096, 32, 10, 32768, 65536, 32768, 32768)
    n = C.c_int32(1)
    nd = C.addressof(n)
    ok = [pool, 4096, 4, 4096, nd, 4, 4096, 4096, 4, 4096, nd, 4, 4096, 0, 0]

    def call(**kw):
        a = list(ok)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return cascade.cascade_pack_unpack(*a)
    assert call(a1=0) == cascade.EINVAL                  # pack staging missing
    assert call(a7=4100) == cascade.EINVAL               # unpack staging misaligned
    assert call(a6=0) == cascade.EINVAL                  # pack hazards missing
    assert call(a12=0) == cascade.EINVAL                 # unpack hazards missing
    assert call(a5=-1) == cascade.EINVAL
    assert call(a0=cascade.KvPool(4096, 2, 10, 24, 0, 0, 0)) == cascade.EINVAL
    assert call(a5=0, a11=0) == cascade.OK               # nothing to launch
    assert call(a5=0, a6=0, a11=0, a12=0) == cascade.OK  # empty lists need no hazards


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(cascade, "_lib", None)
    monkeypatch.setattr(cascade, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        cascade.load()


def test_reclaim_workspace_size(lib):
    prev = 0
    for n in [0, 1, 2048, 2049, 95367, 1 << 22, 1 << 30]:
        b = cascade.cascade_reclaim_workspace_bytes(n)
        assert b % 256 == 0 and b >= prev and b > 0
        prev = b
    assert cascade.cascade_reclaim_workspace_bytes(-1) == 0
    assert cascade.cascade_reclaim_workspace_bytes((1 << 30) + 1) == 0


def test_reclaim_host_checks(lib):
    fake = 4096  # never dereferenced: every case below fails a host-side check
    ws_bytes = cascade.cascade_reclaim_workspace_bytes(100)
    tab = cascade.TierTable(100, fake, fake, fake)

    def call(tier=0, table=tab, need=10, inc=0, n_inc=0, max_in=0, out=fake, n_out=fake,
             max_out=10, freed=fake, placed=0, index=0, cap=0, ws=fake * 2, wsb=ws_bytes,
             status=fake):
        return cascade.cascade_tier_reclaim(tier, table, need, inc, n_inc, max_in, out, n_out,
                                            max_out, freed, placed, index, cap, ws, wsb, status, 0)

    E = cascade.EINVAL
    assert call(tier=3) == E
    assert call(tier=-1) == E
    assert call(need=-1) == E
    assert call(status=0) == E
    assert call(table=cascade.TierTable(-1, fake, fake, fake)) == E
    assert call(table=cascade.TierTable(100, 0, fake, fake)) == E
    assert call(table=cascade.TierTable(100, fake + 8, fake, fake)) == E  # misaligned
    assert call(table=cascade.TierTable(100, fake, fake + 8, fake)) == E
    assert call(table=cascade.TierTable(100, fake, fake, fake + 1)) == E
    assert call(max_in=5) == E                       # incoming buffers missing
    assert call(max_in=5, inc=fake, n_inc=fake) == E  # placed missing
    assert call(max_out=9) == E                      # room for need demotions
    assert call(n_out=0) == E
    assert call(freed=0) == E
    assert call(index=fake, cap=100) == E            # capacity not a power of two
    assert call(index=fake + 8, cap=1024) == E       # misaligned index
    assert call(ws=0) == E
    assert call(ws=fake + 16) == E                   # workspace not 256-byte aligned
    assert call(wsb=ws_bytes - 1) == E
    assert call(need=2**31 - 1, max_in=1, inc=fake, n_inc=fake, placed=fake) == E
    # NVMe demotes nothing: no outgoing room needed, but the rest still checked
    assert call(tier=2, max_out=0, out=0, n_out=0, wsb=ws_bytes - 1) == E


def test_reclaim_chain_host_checks(lib):
    fake = 4096  # never dereferenced: every case below fails a host-side check
    n = [100, 200, 300]
    wsb = cascade.cascade_tier_chain_workspace_bytes(n)
    assert wsb == sum(cascade.cascade_reclaim_workspace_bytes(x) for x in n)
    assert cascade.cascade_tier_chain_workspace_bytes([100, -1, 300]) == 0
    assert cascade.cascade_tier_chain_workspace_bytes([100, 200, (1 << 30) + 1]) == 0

    def chain(**kw):
        c = cascade.TierChain()
        for t in range(3):
            c.table[t] = cascade.TierTable(n[t], fake, fake, fake)
            c.need[t] = 10
            c.freed[t] = fake
            c.placed[t] = fake if t > 0 else 0
        for t in range(2):
            c.outgoing[t] = fake
            c.n_outgoing_dev[t] = fake
        c.max_outgoing[0] = 10
        c.max_outgoing[1] = 20
        for k, v in kw.items():
            t, f, x = v
            getattr(c, f)[t] = x
        return c

    def call(c=None, ws=fake * 2, b=wsb, status=fake):
        return cascade.cascade_tier_reclaim_chain(c if c is not None else chain(), 0, 0, ws, b,
                                                  status, 0)

    E = cascade.EINVAL
    assert call(b=wsb - 1) == E                     # room for three workspaces
    assert call(ws=0) == E
    assert call(ws=fake + 16) == E                  # not 256-byte aligned
    assert call(status=0) == E
    assert call(chain(a=(1, "need", -1))) == E
    assert call(chain(a=(0, "max_outgoing", 9))) == E   # tier 0: room for its demotions
    assert call(chain(a=(1, "max_outgoing", 19))) == E  # tier 1: need + tier 0's demotions
    assert call(chain(a=(2, "placed", 0))) == E          # tier 2 receives tier 1's demotions
    assert call(chain(a=(2, "freed", 0))) == E
    bad = chain()
    bad.table[1] = cascade.TierTable(200, fake + 8, fake, fake)  # misaligned
    assert call(bad) == E
