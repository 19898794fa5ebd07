"""Host check of the matrix-core product's launch planner (csrc/gemm_plan.h), CPU only.

A product whose reduction is split writes one partial tile (and row sums) per slice into a
caller-given workspace; the planner must never launch more slices than that workspace holds.
The variant pass once sized its workspace for a full chunk only and faulted the GPU on a short
last chunk whose products split further; the planner now clamps the split to the workspace and
the pass sizes it for both chunk lengths. The header is compiled for the host with g++ and its
plans are checked here over the training, variant and benchmark shapes; nothing touches a GPU.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_09486_amd", "csrc")

PROGRAM = r"""
#include "gemm_plan.h"
#include <cstdio>
#include <cstring>
using namespace enova;
int main() {
    char op[8];
    while (std::scanf("%7s", op) == 1) {
        if (!std::strcmp(op, "P")) {           // m n k may_split work_floats -> tm tn kc used
            int m, n, k, may; long long ws;
            std::scanf("%d %d %d %d %lld", &m, &n, &k, &may, &ws);
            GemmPlan p = gemm_plan(m, n, k, may != 0, ws);
            std::printf("%d %d %d %d\n", p.tm, p.tn, p.kc, p.used);
        } else if (!std::strcmp(op, "S")) {    // m n k -> splits, workspace, slice floats
            int m, n, k;
            std::scanf("%d %d %d", &m, &n, &k);
            std::printf("%d %lld %lld\n", gemm_splits(m, n, k), (long long)gemm_workspace_floats(m, n, k),
                        (long long)gemm_slice_floats(m, n));
        } else if (!std::strcmp(op, "V")) {    // D H L n_windows -> chunk, last rows, workspace
            int D, H, L; long long N;
            std::scanf("%d %d %d %lld", &D, &H, &L, &N);
            int B = variants_chunk(D, N), last = variants_last_rows(N, B);
            std::printf("%d %d %lld\n", B, last, (long long)variants_gemm_workspace(B, last, D, H, L));
        } else if (!std::strcmp(op, "R")) {    // m n k a_k b_k may_split work -> kind tm tn unit kc used
            int m, n, k, ak, bk, may; long long ws;
            std::scanf("%d %d %d %d %d %d %lld", &m, &n, &k, &ak, &bk, &may, &ws);
            RsPlan p = gemm_rs_plan(m, n, k, ak != 0, bk != 0, true, true, may != 0, ws);
            RsShape sh = rs_shape(p.kind);
            std::printf("%d %d %d %d %d %d\n", p.kind, sh.tm, sh.tn, p.kind ? rs_k_unit(p.kind) : 0, p.kc, p.used);
        } else if (!std::strcmp(op, "T")) {    // B D H L -> training workspace
            int B, D, H, L;
            std::scanf("%d %d %d %d", &B, &D, &H, &L);
            std::printf("%lld\n", (long long)train_gemm_workspace(B, D, H, L));
        } else if (!std::strcmp(op, "G")) {    // B D H L which -> m n k, its own workspace
            int B, D, H, L, w, m, n, k;
            std::scanf("%d %d %d %d %d", &B, &D, &H, &L, &w);
            train_grad_shape(B, D, H, L, w, m, n, k);
            std::printf("%d %d %d %lld\n", m, n, k, (long long)train_grad_workspace(B, D, H, L, w));
        }
        std::fflush(stdout);
    }
    return 0;
}
"""


class Planner:
    def __init__(self, exe):
        self.exe = exe

    def run(self, lines):
        r = subprocess.run([self.exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                           check=True, timeout=60)
        return [list(map(int, ln.split())) for ln in r.stdout.strip().splitlines()]


@pytest.fixture(scope="module")
def planner():
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not available")
    d = tempfile.mkdtemp()
    try:
        src = os.path.join(d, "plan.cpp")
        exe = os.path.join(d, "plan")
        with open(src, "w") as f:
            f.write(PROGRAM)
        subprocess.run([gxx, "-std=c++17", "-O1", "-Wall", "-I", CSRC, src, "-o", exe], check=True)
        yield Planner(exe)
    finally:
        shutil.rmtree(d, ignore_errors=True)


def _check_plans(planner, shapes, ws, may=1):
    """Every plan covers k exactly with whole slices and its partials fit the workspace."""
    out = planner.run([f"P {m} {n} {k} {may} {ws}" for m, n, k in shapes])
    slice_f = planner.run([f"S {m} {n} {k}" for m, n, k in shapes])
    for (m, n, k), (tm, tn, kc, used), (_, _, per) in zip(shapes, out, slice_f):
        assert used >= 1 and kc >= 1
        assert (used - 1) * kc < max(k, 1) <= used * kc, (m, n, k, kc, used)
        if used > 1:
            assert kc % 32 == 0, (m, n, k, kc)
            assert used * per <= ws, f"{(m, n, k)}: {used} slices x {per} floats > workspace {ws}"
        assert tm in (32, 128) and tn in (32, 128)
    return out


# (D, H, L) of the five detector shapes and of the variant tests
DET = [(256, 32, 16), (512, 64, 16), (2048, 128, 16), (8192, 256, 16), (1024, 128, 16),
       (64 * 5, 128, 16), (32 * 3, 64, 8), (16 * 12, 32, 4)]


def _variant_shapes(rows, D, H, L):
    return [(rows, H, D), (rows, 2 * L, H), (rows, H, L), (rows, D, H)]


@pytest.mark.parametrize("D,H,L", DET)
def test_variant_pass_products_fit_their_workspace(planner, D, H, L):
    # n_windows around the chunk length, the c5 benchmark's window count and its old fault case
    chunk = planner.run([f"V {D} {H} {L} 1000000000"])[0][0]
    counts = {1, 7, 255, 256, 257, 12842, chunk - 1, chunk, chunk + 1, 2 * chunk + 12842, 3 * chunk + 100,
              134951466}
    for N in sorted(c for c in counts if c >= 1):
        B, last, ws = planner.run([f"V {D} {H} {L} {N}"])[0]
        assert 1 <= last <= B and (N - last) % B == 0
        assert B == min(N, max(256, min((1 << 28) // D, 262144)))
        for rows in {B, last}:
            _check_plans(planner, _variant_shapes(rows, D, H, L), ws)


def test_short_last_chunk_is_clamped_to_a_full_chunk_workspace(planner):
    """The fault's mechanism: c5's variant pass (D = 1024, H = 128, L = 16) in full chunks needs
    no split workspace, but a short last chunk (2000 windows here) has so few output tiles that its
    encoder product wants several slices; with a workspace sized for the full chunk only, the
    planner must split less instead of writing past the workspace."""
    D, H, L = 1024, 128, 16
    B = planner.run([f"V {D} {H} {L} 1000000000"])[0][0]
    _, _, ws_full_only = planner.run([f"V {D} {H} {L} {B}"])[0]
    wanted = planner.run([f"S 2000 {H} {D}"])[0]
    assert wanted[0] > 1 and wanted[0] * wanted[2] > ws_full_only      # it wants more than there is
    out = _check_plans(planner, _variant_shapes(2000, D, H, L), ws_full_only)
    assert out[0][3] * wanted[2] <= ws_full_only or out[0][3] == 1
    # the pass itself sizes the workspace for the last chunk too, so there it splits as it wants
    _, last, ws = planner.run([f"V {D} {H} {L} {B + 2000}"])[0]
    assert last == 2000
    out = _check_plans(planner, _variant_shapes(2000, D, H, L), ws)
    assert out[0][3] == wanted[0]
    # no workspace at all: nothing splits
    out = _check_plans(planner, _variant_shapes(2000, D, H, L), 0)
    assert all(p[3] == 1 for p in out)
    # a product that may not split (a reduction epilogue) never does, whatever the workspace
    out = _check_plans(planner, _variant_shapes(300, D, H, L), 1 << 40, may=0)
    assert all(p[3] == 1 for p in out)


@pytest.mark.parametrize("B", [1, 31, 32, 33, 127, 128, 500, 4096, 8192, 8193, 65536])
@pytest.mark.parametrize("D,H,L", [(1024, 128, 16), (256, 32, 16), (8192, 256, 16), (12, 5, 3)])
def test_training_products_fit_their_workspace(planner, B, D, H, L):
    ws = planner.run([f"T {B} {D} {H} {L}"])[0][0]
    shapes = [(B, H, D), (B, 2 * L, H), (B, H, L), (B, D, H), (D, H, B), (B, H, D), (H, L, B), (B, L, H),
              (2 * L, H, B), (B, H, 2 * L), (H, D, B)]
    out = _check_plans(planner, shapes, ws)
    # with the step's own workspace every product splits as far as it wants
    want = planner.run([f"S {m} {n} {k}" for m, n, k in shapes])
    for (m, n, k), p, w in zip(shapes, out, want):
        assert p[3] <= w[0]
        if w[0] > 1:
            assert p[3] > 1, (m, n, k)


@pytest.mark.parametrize("B", [1, 31, 32, 33, 127, 128, 500, 4096, 8192, 8193, 65536])
@pytest.mark.parametrize("D,H,L", [(1024, 128, 16), (256, 32, 16), (8192, 256, 16), (12, 5, 3)])
def test_weight_gradient_products_fit_their_own_regions(planner, B, D, H, L):
    """The four weight-gradient products keep their slices until the Adam step sums them, each in
    a workspace region of its own: the region must hold every slice the product is planned to
    write (on either kernel), and must not make it split less than with the shared workspace."""
    shared = planner.run([f"T {B} {D} {H} {L}"])[0][0]
    expect = [(D, H, B), (H, L, B), (2 * L, H, B), (H, D, B)]
    for w in range(4):
        m, n, k, ws = planner.run([f"G {B} {D} {H} {L} {w}"])[0]
        assert (m, n, k) == expect[w]
        assert ws <= shared
        mine = _check_plans(planner, [(m, n, k)], ws)[0]
        assert mine == _check_plans(planner, [(m, n, k)], shared)[0]
        rs = _check_rs(planner, [(m, n, k, 0, 0)], ws)[0]
        assert rs == _check_rs(planner, [(m, n, k, 0, 0)], shared)[0]


# the step's products as (m, n, k, A k-contiguous, B k-contiguous), in launch order
def _train_layouts(B, D, H, L):
    return [(B, H, D, 1, 1), (B, 2 * L, H, 1, 1), (B, H, L, 1, 1), (B, D, H, 1, 1), (D, H, B, 0, 0),
            (B, H, D, 1, 0), (H, L, B, 0, 0), (B, L, H, 1, 0), (2 * L, H, B, 0, 0), (B, H, 2 * L, 1, 0),
            (H, D, B, 0, 0)]


def _check_rs(planner, layouts, ws, may=1):
    out = planner.run([f"R {m} {n} {k} {a} {b} {may} {ws}" for m, n, k, a, b in layouts])
    for (m, n, k, a, b), (kind, tm, tn, unit, kc, used) in zip(layouts, out):
        if kind == 0:
            continue
        assert kind in (1, 3)
        assert m % tm == 0 and n % tn == 0, (m, n, k, kind)
        assert kc * used == k and kc % unit == 0, (m, n, k, kc, used, unit)
        if kind == 1:
            assert a == 1 and used == 1 and k >= 512
            assert ((m + 127) // 128) * ((n + 127) // 128) < 128, (m, n, k)
        if kind == 3:
            assert a == 0 and b == 0
        if used > 1:
            assert may and used * (m * n + m) <= ws, (m, n, k, used, ws)
    return out


@pytest.mark.parametrize("B", [1, 32, 64, 500, 512, 3000, 4096, 8192, 65536])
@pytest.mark.parametrize("D,H,L", [(1024, 128, 16), (512, 128, 16), (256, 32, 16), (8192, 256, 16), (102, 70, 16)])
def test_register_streamed_plans_cover_whole_tiles(planner, B, D, H, L):
    ws = planner.run([f"T {B} {D} {H} {L}"])[0][0]
    _check_rs(planner, _train_layouts(B, D, H, L), ws)
    _check_rs(planner, _train_layouts(B, D, H, L), 0, may=0)


def test_register_streamed_plans_of_the_training_workload(planner):
    """c5's training shape (D = 1024, H = 128, L = 16, B = 8192): the encoder, dJ/da2 and the two
    large weight gradients take the register-streamed kernel (the weight gradients split their
    8192-long reduction over blocks); the decoder output (a reduction of 128) and the thin
    products stay on the LDS-tiled kernel."""
    B, D, H, L = 8192, 1024, 128, 16
    ws = planner.run([f"T {B} {D} {H} {L}"])[0][0]
    out = _check_rs(planner, _train_layouts(B, D, H, L), ws)
    kinds = [o[0] for o in out]
    # the variant pass's encoder over a full chunk of 262144 windows keeps the LDS-tiled kernel
    assert _check_rs(planner, [(262144, H, D, 1, 1)], 0, may=0)[0][0] == 0
    assert kinds[0] == 1 and kinds[5] == 1 and kinds[3] == 0      # encoder, dJ/da2; decoder output
    assert kinds[4] == 3 and kinds[10] == 3                       # dWd2, dW1
    assert out[4][5] == 8 and out[10][5] == 8
    assert kinds[1] == kinds[2] == kinds[6] == kinds[7] == kinds[8] == kinds[9] == 0
