"""The C-ABI library on the host (no GPU): it loads, exports every entry point
include/sn.h declares, and rejects invalid arguments before any launch.

Every call here fails validation (or is an N == 0 no-op), so nothing touches a
device; the pointers are never dereferenced.
"""
import ctypes
import os
import re

import pytest

import paper_2506_01260_amd as sn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sn.h")
FAKE = 0x7F0000000000            # a 256-byte-aligned address that is never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(sn_\w+)\s*\(", text, flags=re.M)))


def test_library_loads_and_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 10
    L = ctypes.CDLL(sn.LIB_PATH)
    for name in names:
        assert hasattr(L, name), f"{name} declared in sn.h but not exported"
    assert set(names) == set(sn._SIGNATURES), "binding and header disagree"
    assert sn.sn_version().endswith("gfx950")


def test_status_strings():
    L = sn.lib()
    assert L.sn_status_string(0) == b"SN_OK"
    for code, name in sn.STATUS.items():
        assert L.sn_status_string(code).decode() == name


def test_packed_and_workspace_sizes():
    assert sn.sn_basis_packed_bytes(4096, 40, 1) > 4096 * 40 * 4
    assert sn.sn_basis_packed_bytes(4096, 40, 1) % 256 == 0
    assert sn.sn_basis_packed_bytes(4096, 0, 1) == 0
    assert sn.sn_basis_packed_bytes(8, 9, 1) == 0          # k > d
    assert sn.sn_basis_packed_bytes(4096, 40, 7) == 0      # bad dtype
    assert sn.sn_basis_packed_bytes(4096, 257, 1) == 0     # k > SN_MAX_K
    assert sn.lib().sn_project_weights_workspace_bytes(4096, 40, 1, 4096) > 0


def _compress(**over):
    a = dict(basis=FAKE, d=256, k=8, dt=1, X=FAKE + (1 << 20), N=16, ldx=256, tok=FAKE + (2 << 20),
             E=FAKE + (3 << 20), vocab=10, lde=256, pos=None, P=None, n_pos=0, ldp=0,
             seq_len=0, C=FAKE + (8 << 20), ldc=8, err=None, stream=None)
    a.update(over)
    return sn.lib().sn_compress(a["basis"], a["d"], a["k"], a["dt"], a["X"], a["N"], a["ldx"],
                                a["tok"], a["E"], a["vocab"], a["lde"], a["pos"], a["P"],
                                a["n_pos"], a["ldp"], a["seq_len"], a["C"], a["ldc"], a["err"],
                                a["stream"])


@pytest.mark.parametrize("over,code", [
    (dict(basis=None), 1),
    (dict(basis=FAKE + 16), 4),                 # packed basis not 256-aligned
    (dict(dt=5), 3),
    (dict(k=0), 2), (dict(k=300, d=512), 8), (dict(k=9, d=8, ldx=8), 2),
    (dict(N=-1), 2), (dict(ldx=255), 2), (dict(ldc=7), 2),
    (dict(tok=None), 1),                         # E given without ids
    (dict(vocab=0), 2), (dict(lde=100), 2),
    (dict(P=FAKE + (4 << 20), n_pos=4, ldp=256, seq_len=0), 2),   # default pos needs seq_len
    (dict(P=FAKE + (4 << 20), n_pos=4, ldp=256, seq_len=5), 2),   # seq_len > n_pos
    (dict(X=None), 1), (dict(C=None), 1),
    (dict(X=FAKE + 1), 4),                       # misaligned bf16 pointer
    (dict(C=FAKE + (1 << 20) + 64), 5),          # C overlaps X
    (dict(C=FAKE + (3 << 20)), 5),               # C overlaps E
    (dict(C=FAKE + 512), 5),                     # C overlaps the packed basis
])
def test_compress_rejects_invalid_arguments(over, code):
    assert _compress(**over) == code
    assert sn.lib().sn_last_error().decode() != ""


def test_empty_batch_returns_ok_without_launch():
    assert _compress(N=0, X=None, C=None) == 0


def test_decompress_and_projection_validation():
    L = sn.lib()
    # decompress: output overlapping its input C
    st = L.sn_decompress(FAKE, 256, 8, 1, FAKE + (1 << 20), 16, 8, None, None, 0, 0, None, None,
                         0, 0, 0, FAKE + (1 << 20), 256, None, None)
    assert st == 5
    st = L.sn_grad_compress(FAKE, 256, 8, 1, FAKE + (1 << 20), 16, 100, FAKE + (8 << 20), 8, None)
    assert st == 2                                # ldg < d
    # projection: workspace too small, misaligned, overlapping, m == 0
    need = L.sn_project_weights_workspace_bytes(256, 8, 1, 64)
    st = L.sn_project_weights(FAKE, 256, 8, 1, FAKE + (1 << 20), 64, 64, FAKE + (8 << 20),
                              need - 1, None)
    assert st == 9
    st = L.sn_project_weights(FAKE, 256, 8, 1, FAKE + (1 << 20), 64, 64, FAKE + (8 << 20) + 8,
                              need, None)
    assert st == 4
    st = L.sn_project_weights(FAKE, 256, 8, 1, FAKE + (1 << 20), 64, 64, FAKE + (1 << 20),
                              need, None)
    assert st == 5
    assert L.sn_project_weights(FAKE, 256, 8, 1, None, 0, 0, None, 0, None) == 0
    # pack: too small a buffer, misaligned target
    assert L.sn_basis_pack(FAKE + (1 << 20), 256, 8, 8, 1, FAKE, 100, None) == 9
    assert L.sn_basis_pack(FAKE + (1 << 20), 256, 8, 8, 1, FAKE + 8, 1 << 20, None) == 4
    assert L.sn_basis_pack(FAKE + (1 << 20), 256, 8, 4, 1, FAKE, 1 << 20, None) == 2


def test_binding_rejects_host_tensors():
    import torch
    U = torch.zeros(64, 8, dtype=torch.bfloat16)
    with pytest.raises(sn.SnError):
        sn.sn_basis_pack(U)


def test_projected_tables_validation():
    L = sn.lib()
    # layout: fp32 rows padded to 16 * ceil(k / 16); P U section 256-byte aligned
    assert L.sn_embed_projected_bytes(40, 10, 4) == 2048 + 768     # kp = 48
    assert L.sn_embed_projected_bytes(16, 3, 0) == 256
    assert L.sn_embed_projected_bytes(40, 0, 0) == 0
    assert L.sn_embed_projected_bytes(0, 10, 4) == 0
    assert L.sn_embed_projected_bytes(40, -1, 4) == 0
    need = L.sn_embed_projected_bytes(8, 10, 4)
    E, P, out = FAKE + (1 << 20), FAKE + (2 << 20), FAKE + (8 << 20)
    ok = dict(E=E, vocab=10, lde=256, P=P, n_pos=4, ldp=256, out=out, nbytes=need)

    def embed(**over):
        a = dict(ok)
        a.update(over)
        return L.sn_embed_project(FAKE, 256, 8, 1, a["E"], a["vocab"], a["lde"], a["P"],
                                  a["n_pos"], a["ldp"], a["out"], a["nbytes"], None)
    assert embed(E=None) == 1                     # vocab > 0 without E
    assert embed(P=None) == 1
    assert embed(vocab=0) == 1                    # E given with vocab == 0
    assert embed(lde=100) == 2
    assert embed(nbytes=need - 1) == 9
    assert embed(out=out + 64) == 4
    assert embed(out=E) == 5                      # overlaps E
    assert embed(out=FAKE) == 5                   # overlaps the basis
    assert embed(E=None, vocab=0, P=None, n_pos=0, out=None, nbytes=0) == 0

    def comp(**over):
        a = dict(X=FAKE + (3 << 20), N=16, ldx=256, tok=FAKE + (4 << 20), pos=None, seq_len=4,
                 proj=out, vocab=10, n_pos=4, C=FAKE + (5 << 20), ldc=8)
        a.update(over)
        return L.sn_compress_projected(FAKE, 256, 8, 1, a["X"], a["N"], a["ldx"], a["tok"],
                                       a["pos"], a["seq_len"], a["proj"], a["vocab"],
                                       a["n_pos"], a["C"], a["ldc"], None, None)
    assert comp(proj=None) == 1
    assert comp(proj=out + 16) == 4
    assert comp(tok=None) == 1
    assert comp(seq_len=0) == 2 and comp(seq_len=5) == 2
    assert comp(ldc=7) == 2 and comp(ldx=255) == 2
    assert comp(C=out) == 5                       # C overlaps the tables
    assert comp(C=FAKE + (3 << 20)) == 5          # C overlaps X
    assert comp(N=0, X=None, C=None) == 0


def test_grassmann_sizes_and_validation():
    L = sn.lib()
    # state: 256-byte head, then Y (d x k float64)
    assert L.sn_grassmann_state_bytes(256, 8) == 256 + 256 * 8 * 8
    assert L.sn_grassmann_state_bytes(256, 129) == 0            # k > 128
    assert L.sn_grassmann_state_bytes(8, 9) == 0
    ws = L.sn_grassmann_workspace_bytes(256, 8, 1, 512)
    assert ws > 0 and ws >= L.sn_grassmann_workspace_bytes(256, 8, 1, 0) > 0
    assert L.sn_grassmann_workspace_bytes(256, 8, 7, 512) == 0
    state, w = FAKE + (16 << 20), FAKE + (24 << 20)
    G, C = FAKE + (1 << 20), FAKE + (8 << 20)

    def acc(**over):
        a = dict(basis=FAKE, d=256, k=8, dt=1, G=G, N=512, ldg=256, C=C, ldc=8, su=1,
                 state=state, ws=w, nbytes=ws)
        a.update(over)
        return L.sn_grassmann_accumulate(a["basis"], a["d"], a["k"], a["dt"], a["G"], a["N"],
                                         a["ldg"], a["C"], a["ldc"], a["su"], a["state"],
                                         a["ws"], a["nbytes"], None)
    assert acc(basis=None) == 1
    assert acc(state=None) == 1 and acc(state=state + 8) == 4
    assert acc(k=129, d=512, ldg=512, ldc=129) == 8                # k above the update's limit
    assert acc(ldg=100) == 2 and acc(ldc=7) == 2
    assert acc(G=None) == 1 and acc(G=G + 1) == 4
    assert acc(ws=None) == 1 and acc(ws=w + 16) == 4 and acc(nbytes=ws - 1) == 9
    assert acc(C=G) == 5                                           # Cg overlaps G
    assert acc(state=G) == 5                                       # state overlaps G
    assert acc(ws=FAKE) == 5                                       # workspace overlaps the basis
    assert acc(N=0, G=None) == 0

    sw = L.sn_grassmann_workspace_bytes(256, 8, 1, 0)

    def step(**over):
        a = dict(basis=FAKE, state=state, eta=0.1, U=C, ldu=8, odt=0, ws=w, nbytes=sw, err=None)
        a.update(over)
        return L.sn_grassmann_step(a["basis"], 256, 8, 1, a["state"], a["eta"], a["U"], a["ldu"],
                                   a["odt"], a["ws"], a["nbytes"], a["err"], None)
    assert step(U=None) == 1 and step(state=None) == 1
    assert step(eta=-1.0) == 2 and step(eta=float("nan")) == 2 and step(eta=float("inf")) == 2
    assert step(ldu=4) == 2 and step(odt=5) == 3
    assert step(nbytes=sw - 1) == 9
    assert step(U=state) == 5 and step(U=w) == 5 and step(U=FAKE) == 5
    assert step(err=C + (1 << 20) + 2) == 4
    assert L.sn_grassmann_reset(None, 256, 8, None) == 1
    assert L.sn_grassmann_reset(state + 64, 256, 8, None) == 4
    assert L.sn_grassmann_reset(state, 256, 300, None) == 2


def test_adamw_sizes_and_validation():
    L = sn.lib()
    assert L.sn_adamw_workspace_bytes(4096, 14336) >= (4096 // 64 + 1) * 14336 * 4
    assert L.sn_adamw_workspace_bytes(-1, 8) == 0
    W, G, M, V, w = (FAKE + (i << 24) for i in range(1, 6))
    need = L.sn_adamw_workspace_bytes(64, 32)

    def step(**over):
        a = dict(W=W, ldw=32, G=G, ldg=32, dt=1, M=M, V=V, ldm=32, rows=64, cols=32, t=1,
                 lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, wd=0.0, sub=1, ws=w, nbytes=need)
        a.update(over)
        return L.sn_adamw_step(a["W"], a["ldw"], a["G"], a["ldg"], a["dt"], a["M"], a["V"],
                               a["ldm"], a["rows"], a["cols"], a["t"], a["lr"], a["b1"], a["b2"],
                               a["eps"], a["wd"], a["sub"], a["ws"], a["nbytes"], None)
    assert step(dt=4) == 3
    assert step(t=0) == 2 and step(b1=1.0) == 2 and step(b2=-0.1) == 2
    assert step(lr=float("nan")) == 2 and step(eps=-1.0) == 2 and step(wd=float("inf")) == 2
    assert step(ldw=16) == 2 and step(ldm=31) == 2
    assert step(W=None) == 1 and step(M=None) == 1
    assert step(W=W + 1) == 4 and step(M=M + 2) == 4
    assert step(ws=None) == 1 and step(nbytes=need - 1) == 9 and step(ws=w + 64) == 4
    assert step(G=W) == 5 and step(V=M + 64) == 5 and step(ws=V) == 5
    assert step(rows=0, W=None, G=None) == 0


def test_embed_lowrank_validation():
    L = sn.lib()
    need = L.sn_embed_lowrank_workspace_bytes(256, 8, 1, 512, 100)
    assert need > 512 * 16 * 4 and L.sn_embed_lowrank_workspace_bytes(256, 8, 1, 512, 0) == 0
    CS, tok, E, X0, w, g = (FAKE + (i << 24) for i in range(1, 7))

    def fwd(**over):
        a = dict(CS=CS, vocab=100, ldcs=8, tok=tok, E=E, lde=256, X0=X0, N=512, ldx=256, ws=w,
                 nbytes=need)
        a.update(over)
        return L.sn_embed_lowrank_forward(FAKE, 256, 8, 1, a["CS"], a["vocab"], a["ldcs"],
                                          a["tok"], a["E"], a["lde"], None, None, 0, 0, 0,
                                          a["X0"], a["N"], a["ldx"], None, a["ws"], a["nbytes"],
                                          None)
    assert fwd(CS=None) == 1 and fwd(tok=None) == 1 and fwd(X0=None) == 1
    assert fwd(ldcs=4) == 2 and fwd(ldx=100) == 2 and fwd(vocab=0) == 2
    assert fwd(nbytes=need - 1) == 9 and fwd(ws=w + 8) == 4
    assert fwd(X0=CS) == 5 and fwd(ws=X0) == 5
    assert fwd(N=0, X0=None) == 0

    def bwd(**over):
        a = dict(dX=X0, N=512, ldg=256, tok=tok, vocab=100, g=g, ldgc=8, ws=w, nbytes=need)
        a.update(over)
        return L.sn_embed_lowrank_backward(FAKE, 256, 8, 1, a["dX"], a["N"], a["ldg"], a["tok"],
                                           a["vocab"], a["g"], a["ldgc"], None, a["ws"],
                                           a["nbytes"], None)
    assert bwd(dX=None) == 1 and bwd(g=None) == 1 and bwd(tok=None) == 1
    assert bwd(ldg=10) == 2 and bwd(ldgc=7) == 2 and bwd(vocab=0) == 2
    assert bwd(g=g + 2) == 4 and bwd(nbytes=need - 1) == 9
    assert bwd(g=X0) == 5 and bwd(ws=tok) == 5
    assert bwd(N=0, dX=None) == 0


def test_project_multi_validation():
    L = sn.lib()
    M = (ctypes.c_int64 * 3)(512, 256, 300)
    need = L.sn_project_weights_multi_workspace_bytes(256, 8, 1, 3, M)
    assert need >= L.sn_project_weights_workspace_bytes(256, 8, 1, 512)
    assert L.sn_project_weights_multi_workspace_bytes(256, 8, 1, 17, M) == 0
    W = (ctypes.c_void_p * 3)(FAKE + (1 << 24), FAKE + (2 << 24), FAKE + (3 << 24))
    LD = (ctypes.c_int64 * 3)(512, 256, 300)
    ws = FAKE + (8 << 24)

    def call(count=3, Wp=W, Mp=M, LDp=LD, w=ws, nbytes=need):
        return L.sn_project_weights_multi(FAKE, 256, 8, 1, count, Wp, Mp, LDp, w, nbytes, None)
    assert call(count=17) == 2 and call(count=-1) == 2
    assert call(Wp=None) == 1 and call(w=None) == 1
    assert call(nbytes=need - 1) == 9 and call(w=ws + 64) == 4
    bad_ld = (ctypes.c_int64 * 3)(512, 255, 300)
    assert call(LDp=bad_ld) == 2
    overlapping = (ctypes.c_void_p * 3)(FAKE + (1 << 24), FAKE + (1 << 24) + 1024, FAKE + (3 << 24))
    assert call(Wp=overlapping) == 5
    assert call(w=FAKE + (2 << 24)) == 5              # workspace overlaps W[1]
    assert call(count=0) == 0


def test_project_noalloc_validation():
    """The no-alloc projection checks every argument before touching a device,
    including a matrix too large for its static scratch."""
    f = sn.lib().sn_project_weights_noalloc
    W = FAKE + (1 << 20)
    assert f(None, 256, 8, 1, W, 64, 64, None) == 1            # basis NULL
    assert f(FAKE, 256, 8, 1, None, 64, 64, None) == 1         # W NULL
    assert f(FAKE, 256, 8, 1, W, 64, 63, None) == 2            # ldw < m
    assert f(FAKE, 256, 8, 7, W, 64, 64, None) == 3            # dtype
    assert f(FAKE, 256, 8, 1, W + 1, 64, 64, None) == 4        # misaligned bf16 pointer
    assert f(FAKE, 256, 8, 1, None, 0, 0, None) == 0           # m == 0: no-op
    m = 1 << 16
    assert sn.lib().sn_project_weights_workspace_bytes(4096, 40, 1, m) > (128 << 20)
    assert f(FAKE, 4096, 40, 1, W, m, m, None) == 9            # beyond the static scratch
    assert b"static scratch" in sn.lib().sn_last_error()
