"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Tolerance (per output tensor, max |gpu - oracle| / max |oracle|): 1e-4 for
float32 inputs, 2e-2 for bfloat16 inputs with float32 accumulation; the same
bound holds per head (max over the head's elements over the head's own max
|oracle|), so that a wrong head with small outputs cannot hide behind the
others.  Every head of every case is compared, full-size workloads included:
the oracle runs on batches of heads (heads are independent given their
group's B and C).  After every call the workspace's status word must show
that no state wait gave up.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2405_21060_amd.inputs import WORKLOADS, Problem, make_inputs
from tests.ssd_harness import (TOL, announce, elementwise_diag, forward_workspace, head_rel_err, rel_err,
                               run_gpu, to_device, to_f64)

pytestmark = pytest.mark.gpu

HEAD_BATCH = 16   # heads per oracle call (bounds host memory at the 65,536-token workloads)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2405_21060_amd import ssd

    ssd.load_library()  # raises loudly when the HIP library is missing


def compare(inp, y, fin, tag="", heads=None):
    """Every head of ``y`` (b, T, H, P) and ``fin`` (units, H, P, N, or None)
    against the oracle, HEAD_BATCH heads per oracle call; ``heads`` restricts
    the comparison.  Asserts the per-tensor and the per-head bound."""
    p = inp.problem
    tol = TOL[p.dtype]
    hs = list(range(p.nheads)) if heads is None else list(heads)
    dy = ry = df = rf = 0.0
    worst_y = worst_f = diag = 0.0
    finite = True
    for i in range(0, len(hs), HEAD_BATCH):
        hb = hs[i:i + HEAD_BATCH]
        y_ref, fin_ref = oracle.forward_inputs(inp, heads=hb)
        y_gpu = to_f64(y[:, :, hb])
        finite &= bool(np.all(np.isfinite(y_gpu)))
        dy = max(dy, float(np.abs(y_gpu - y_ref).max()))
        ry = max(ry, float(np.abs(y_ref).max()))
        worst_y = max(worst_y, float(head_rel_err(y_gpu, y_ref, 2).max()))
        diag = max(diag, elementwise_diag(y_gpu, y_ref))
        if fin is not None:
            f_gpu = fin[:, hb].cpu().numpy().astype(np.float64)
            finite &= bool(np.all(np.isfinite(f_gpu)))
            df = max(df, float(np.abs(f_gpu - fin_ref).max()))
            rf = max(rf, float(np.abs(fin_ref).max()))
            worst_f = max(worst_f, float(head_rel_err(f_gpu, fin_ref, 1).max()))
    ey = dy / (ry if ry > 0 else 1.0)
    ef = df / (rf if rf > 0 else 1.0)
    announce("  %d heads: rel err y %.3e final %.3e; worst head y %.3e final %.3e; elementwise %.2e "
             "(tol %.0e)" % (len(hs), ey, ef, worst_y, worst_f, diag, tol))
    assert finite
    assert ey <= tol, ey
    assert ef <= tol, ef
    assert worst_y <= tol, worst_y
    assert worst_f <= tol, worst_f


def check(inp, chunk_size=None, heads=None, use_init=True, tag=""):
    p = inp.problem
    announce("%s %s seed-shape b%d T%d H%d P%d N%d G%d Q%s varlen=%s" % (
        tag, p.dtype, p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups,
        chunk_size or p.chunk_size, p.varlen))
    y, fin = run_gpu(inp, chunk_size=chunk_size, use_init=use_init)
    if not use_init:
        inp.initial_states = None
    compare(inp, y, fin, tag, heads)
    return y, fin


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_f32(seed):
    check(make_inputs(WORKLOADS["tiny_f32"], seed), tag="tiny_f32")


@pytest.mark.parametrize("Q", [32, 64, 128, 256])
def test_chunk_sizes_ragged_bf16(Q):
    # several chunks and tiles, ragged last chunk (1000 % Q != 0), G = 2
    p = Problem(2, 1000, 4, 64, 128, 2, Q, "bf16", init_states=True)
    check(make_inputs(p, 5), tag="ragged")


@pytest.mark.parametrize("Q", [32, 64, 256])
def test_chunk_sizes_ragged_f32(Q):
    p = Problem(1, 777, 3, 32, 48, 3, Q, "f32", init_states=True)
    check(make_inputs(p, 6), tag="ragged_f32")


@pytest.mark.parametrize("dims", [(16, 16), (64, 64), (64, 256), (128, 128), (32, 16)])
def test_state_and_head_dims(dims):
    P, N = dims
    p = Problem(1, 600, 2, P, N, 1, 128, "bf16", init_states=True)
    check(make_inputs(p, 7), tag="dims")


def test_single_token_and_short_sequences():
    for T in (1, 2, 17, 255, 256, 257):
        p = Problem(2, T, 3, 16, 32, 1, 256, "f32", init_states=True)
        check(make_inputs(p, T), tag="T=%d" % T)


def test_varlen_small_with_edge_boundaries():
    # boundaries at a chunk edge (64), at a chunk's last token (127 -> 128),
    # length-1 sequences, several sequences inside one chunk
    lens = [64, 63, 1, 1, 70, 5, 3, 200, 1, 40]
    T = sum(lens)
    p = Problem(1, T, 4, 32, 64, 2, 64, "f32", varlen=True, init_states=True)
    inp = make_inputs(p, 8)
    inp.seq_idx = np.repeat(np.arange(len(lens), dtype=np.int32), lens).reshape(1, T)
    inp.nseq = len(lens)
    inp.initial_states = np.random.default_rng(1).standard_normal(
        (len(lens), 4, 32, 64)).astype(np.float32)
    check(inp, tag="varlen_edges_f32")
    check(inp, use_init=False, tag="varlen_edges_noinit")


def test_varlen_bf16_small():
    p = Problem(1, 3000, 8, 64, 128, 4, 256, "bf16", varlen=True, len_lo=1, len_hi=700,
                init_states=True)
    check(make_inputs(p, 9), tag="varlen_bf16_small")


# ---- packed rows given by the device seq_idx on the fused kernels: every
# sequence cut into chunks of its own (the last one partial) from a chunk table
# built on the device
def _packed(lens, H, N, G, seed, init=True):
    T = int(sum(lens))
    p = Problem(1, T, H, 64, N, G, 256, "bf16", varlen=True, init_states=init)
    inp = make_inputs(p, seed)
    inp.seq_idx = np.repeat(np.arange(len(lens), dtype=np.int32), lens).reshape(1, T)
    inp.nseq = len(lens)
    if init:
        inp.initial_states = np.random.default_rng(seed + 1).standard_normal(
            (len(lens), H, 64, N)).astype(np.float32)
    else:
        inp.initial_states = None
    return inp


@pytest.mark.parametrize("lens,H,N,G", [
    # one-token sequences, lengths at and around the chunk length, several
    # sequences inside one chunk, a sequence over three chunks
    ([1, 255, 256, 257, 1, 513, 2, 700, 3], 6, 64, 2),
    ([300, 1, 1, 1, 40, 600, 256], 4, 128, 1),
    ([700, 1, 256, 300, 513], 4, 256, 2),
    # one sequence only, shorter than a chunk
    ([200], 2, 128, 1),
])
def test_fused_packed_rows(lens, H, N, G):
    inp = _packed(lens, H, N, G, 31)
    check(inp, tag="fused_packed")
    check(inp, use_init=False, tag="fused_packed_noinit")


def test_fused_packed_many_sequences():
    """More sequences than the table kernel's workgroup has lanes (1,024), and
    more sequences than chunks."""
    lens = np.random.default_rng(5).integers(1, 4, 1500).tolist() + [600, 900]
    check(_packed(lens, 2, 64, 1, 17), tag="fused_packed_1502_sequences")


@pytest.mark.parametrize("hg", ["1", "4"])
def test_fused_packed_persistent_items(tune, hg):
    """Few persistent workgroups taking many table entries each."""
    tune("max_workgroups", 3)
    tune("heads_per_item", int(hg))
    check(_packed([700, 30, 1, 900, 256, 513], 8, 128, 1, 19), tag="fused_packed_persistent_hg" + hg)


@pytest.mark.parametrize("early", ["1", "2"])
def test_fused_packed_work_order(tune, early):
    """A packed row's chunks taken in table order and by their index within
    their sequence (both forced; few persistent workgroups, 1 and 4 heads per
    item, either state flag): each against the oracle, and the two
    bit-identical (the order moves work between workgroups, not arithmetic)."""
    import torch

    tune("early_state_flag", int(early))
    tune("max_workgroups", 3)
    inp = _packed([700, 30, 1, 900, 256, 513, 1100, 2], 8, 128, 2, 37)
    for hg in (1, 4):
        tune("heads_per_item", hg)
        tune("packed_order", 1)
        y1, f1 = check(inp, tag="packed_table_order_hg%d_e%s" % (hg, early))
        tune("packed_order", 2)
        y2, f2 = check(inp, tag="packed_depth_order_hg%d_e%s" % (hg, early))
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
        assert torch.equal(f1, f2)


def test_fused_packed_one_sequence_equals_plain_row():
    """seq_idx all zero (one sequence) gives exactly the plain row's result:
    the same chunks, the same arithmetic."""
    import torch

    inp = _packed([1300], 8, 128, 2, 23)
    y1, f1 = run_gpu(inp)
    plain = _packed([1300], 8, 128, 2, 23)
    plain.seq_idx = None
    y2, f2 = run_gpu(plain)
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    assert torch.equal(f1, f2)


@pytest.mark.parametrize("early", ["0", "1"])
def test_fused_state_flag_placement(tune, early):
    """Both placements of a chunk's state flag (after its output stage, or
    right after its state is stored) forced on a plain and a packed row, with
    few persistent workgroups so that items wait on each other."""
    tune("early_state_flag", 2 if early == "1" else 1)
    tune("max_workgroups", 5)
    check(make_inputs(Problem(2, 1100, 8, 64, 128, 2, 256, "bf16", init_states=True), 37),
          tag="flag%s_plain" % early)
    check(_packed([300, 1, 700, 256, 90], 4, 64, 1, 41), tag="flag%s_packed" % early)


@pytest.mark.parametrize("early", ["0", "1"])
def test_fused_n256_few_workgroups(tune, early):
    """N = 256 (two column blocks of the state per head) with few persistent
    workgroups, both state-flag placements, 1 and 2 heads per item."""
    tune("early_state_flag", 2 if early == "1" else 1)
    tune("max_workgroups", 3)
    for hg in (1, 2):
        tune("heads_per_item", hg)
        check(make_inputs(Problem(2, 1100, 4, 64, 256, 2, 256, "bf16", init_states=True), 81),
              tag="n256_flag%s_hg%d" % (early, hg))


@pytest.mark.parametrize("N", [64, 128, 256])
def test_fused_right_factor_both_passes(tune, N):
    """The chunk kernel's right factor in a pass of its own and in the
    diagonal block's pass (both forced; late state flag, few persistent
    workgroups, 1 and 5 heads per item): each against the oracle, and the two
    bit-identical (the same products in the same order)."""
    import torch

    tune("early_state_flag", 1)
    tune("max_workgroups", 3)
    inp = make_inputs(Problem(2, 1300, 10, 64, N, 1, 256, "bf16", init_states=True), 53)
    for hg in (1, 5):
        tune("heads_per_item", hg)
        tune("fused_right_factor", 1)
        y1, f1 = check(inp, tag="rf_own_pass_hg%d_n%d" % (hg, N))
        tune("fused_right_factor", 2)
        y2, f2 = check(inp, tag="rf_fused_hg%d_n%d" % (hg, N))
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
        assert torch.equal(f1, f2)


def test_packed_rows_both_device_paths(tune):
    """The general kernels (forced) and the fused ones on one packed row, each
    against the oracle."""
    inp = _packed([100, 400, 1, 256, 800], 4, 128, 2, 29)
    tune("force_general_path", 1)
    check(inp, tag="packed_general_forced")
    tune("force_general_path", 0)
    check(inp, tag="packed_fused")


@pytest.mark.parametrize("shape", [
    # (batch, T, H, N, G): ragged last chunk, N = 64, 3 heads per group (1 head per workgroup)
    (2, 700, 6, 64, 2),
    # one chunk exactly, 2 heads per group
    (1, 256, 4, 128, 2),
    # many chunks, 4 heads per workgroup, several workgroups per (row, chunk)
    (3, 2000, 16, 128, 1),
    # 10 heads per group: 5 heads per work item
    (2, 1300, 10, 128, 1),
    # the state in two column blocks (N 256): ragged, grouped, 5 heads per item
    (2, 700, 6, 256, 2),
    (1, 1300, 10, 256, 1),
])
def test_fused_shapes(shape):
    b, T, H, N, G = shape
    p = Problem(b, T, H, 64, N, G, 256, "bf16", init_states=True)
    check(make_inputs(p, 11), tag="fused")


@pytest.mark.parametrize("hg", ["1", "2", "4", "5"])
def test_fused_persistent_items(tune, hg):
    """Few persistent workgroups, so that each one runs many work items in a row
    (prefetching the next item's operands and the next head's step 1); every
    head is checked."""
    tune("max_workgroups", 3)
    tune("heads_per_item", int(hg))
    p = Problem(2, 1500, 10 if hg == "5" else 8, 64, 128, 1, 256, "bf16", init_states=True)
    check(make_inputs(p, 13), tag="persistent_hg" + hg)


def test_general_path_at_fused_shape(tune):
    """Both device paths at one shape: the general step-by-step kernels (forced)
    and the fused ones must each meet the tolerance against the oracle."""
    p = Problem(2, 1300, 8, 64, 128, 2, 256, "bf16", init_states=True)
    inp = make_inputs(p, 12)
    tune("force_general_path", 1)
    check(inp, tag="general_forced")
    tune("force_general_path", 0)
    check(inp, tag="fused")


def test_deterministic_repeat():
    import torch

    inp = make_inputs(Problem(2, 1024, 8, 64, 128, 1, 256, "bf16"), 3)
    y1, f1 = run_gpu(inp)
    y2, f2 = run_gpu(inp)
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    assert torch.equal(f1, f2)


def test_chunk_size_independence_large():
    """Chunk-size independence at a size beyond the oracle's comfort: the
    block decomposition is exact for any block length (Section 6)."""
    inp = make_inputs(Problem(2, 4096, 16, 64, 128, 1, 256, "bf16"), 4)
    ys = [to_f64(run_gpu(inp, chunk_size=Q)[0]) for Q in (64, 128, 256)]
    for y in ys[:-1]:
        assert rel_err(y, ys[-1]) <= TOL["bf16"]


# Full-size workloads: every configuration of the benchmark's workload list
# (the 130M and 2.7B layers, all six points of the sequence-length and state
# sweep, the packed grouped row) and one GPU's share of the 2.7B layer under
# head and sequence sharding; every head compared.
FULL = ["mamba2_130m", "mamba2_2p7b", "varlen_g8", "sweep_T512_N128", "sweep_T4096_N128",
        "sweep_T16384_N128", "sweep_T65536_N128", "sweep_T16384_N64", "sweep_T16384_N256", "tp8_2p7b",
        "cp8_2p7b"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_all_heads(name):
    check(make_inputs(WORKLOADS[name], 0), tag=name)


# ---- the method's degenerate cases, on the fused shapes and on the general path
EDGE_SHAPES = {
    "fused_n128": Problem(2, 1000, 8, 64, 128, 2, 256, "bf16", init_states=True),
    "fused_n64": Problem(1, 700, 4, 64, 64, 1, 256, "bf16", init_states=True),
    "general_f32": Problem(1, 700, 6, 32, 48, 2, 64, "f32", init_states=True),
    "general_bf16": Problem(2, 500, 4, 16, 32, 2, 128, "bf16", init_states=True),
}


def edge_inputs(p, seed):
    """Head 0: A_log = -inf (A = -0, a = 0: causal linear attention, Section 4);
    head 1: A_log = 12 (the decay underflows to zero within every token: the
    memoryless limit); head 2: dt = 0 on every 7th token and on a run of 300
    tokens across a chunk boundary (such tokens neither decay the state nor
    add to it); the other heads as drawn."""
    inp = make_inputs(p, seed)
    inp.A_log = inp.A_log.copy()
    inp.A_log[0] = -np.inf
    inp.A_log[1] = 12.0
    dt = inp.dt.copy()
    dt[:, ::7, 2] = 0
    dt[:, 200:500, 2] = 0
    inp.dt = dt
    return inp


@pytest.mark.parametrize("sname", sorted(EDGE_SHAPES))
def test_edge_cases(sname):
    inp = edge_inputs(EDGE_SHAPES[sname], 51)
    check(inp, tag="edge/" + sname)


@pytest.mark.parametrize("sname", sorted(EDGE_SHAPES))
def test_no_skip_no_final_states(sname):
    """D = NULL (no skip term) and final_states = NULL (not written): y alone,
    against the oracle with D = 0."""
    inp = edge_inputs(EDGE_SHAPES[sname], 52)
    announce("no D / no final: " + sname)
    y, fin = run_gpu(inp, use_D=False, final=False)
    assert fin is None
    compare(dataclasses.replace(inp, D=np.zeros_like(inp.D)), y, None, "noD/" + sname)


def test_state_wait_timeout_is_reported(tune):
    """A state wait that gives up is reported by ssd_workspace_status and the
    call still completes.  A wait limit of one poll makes every chunk whose
    predecessor has not yet published give up at once (every kernel exits
    normally); with 256 chunks per head on 8 heads, some chunk always starts
    waiting before its predecessor is done.  Then the default limit again:
    the status word of the next call on the same workspace is clean."""
    import torch
    from paper_2405_21060_amd import ssd

    inp = make_inputs(Problem(1, 65536, 8, 64, 128, 1, 256, "bf16"), 61)
    d = to_device(inp)
    ws = forward_workspace(inp)
    tune("state_wait_limit", 1)
    announce("state wait limit 1 poll")
    ssd.forward(d["x"], d["dt"], d["A_log"], d["B"], d["C"], d["D"], workspace=ws)
    torch.cuda.synchronize()
    assert ssd.workspace_status(ws) == ssd.SSD_ERR_STATE_TIMEOUT
    tune("state_wait_limit", 0)
    announce("default state wait limit")
    y, fin = ssd.forward(d["x"], d["dt"], d["A_log"], d["B"], d["C"], d["D"], workspace=ws)
    torch.cuda.synchronize()
    assert ssd.workspace_status(ws) == ssd.SSD_OK
    compare(inp, y, fin, "after timeout", heads=[0, 7])


# ---- packed rows given by host offsets (ssd_forward_varlen): each sequence on
# its slice, on the fused kernel where the shape allows

def check_varlen_host(inp, heads=None, tag=""):
    import torch
    from paper_2405_21060_amd import ssd

    p = inp.problem
    seq = inp.seq_idx.reshape(-1)
    starts = [0] + [int(v) for v in np.flatnonzero(np.diff(seq)) + 1] + [int(seq.size)]
    announce("%s host offsets, %d sequences" % (tag, len(starts) - 1))
    d = to_device(inp)
    prob = ssd.make_problem(1, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
                            ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32, len(starts) - 1)
    ws = torch.empty(max(ssd.ssd_forward_varlen_workspace_bytes(prob, starts), 1), dtype=torch.uint8,
                     device="cuda")
    y, fin = ssd.forward_varlen(d["x"], d["dt"], d["A_log"], d["B"], d["C"], starts, D=d["D"],
                                chunk_size=p.chunk_size, initial_states=d["initial_states"], workspace=ws)
    torch.cuda.synchronize()
    assert ssd.workspace_status(ws) == ssd.SSD_OK
    compare(inp, y, fin, tag, heads)


def test_varlen_host_offsets_small():
    p = Problem(1, 3000, 8, 64, 128, 4, 256, "bf16", varlen=True, len_lo=1, len_hi=700, init_states=True)
    check_varlen_host(make_inputs(p, 9), tag="varlen_bf16_small")
    p = Problem(1, 700, 4, 32, 64, 2, 64, "f32", varlen=True, len_lo=1, len_hi=200, init_states=True)
    check_varlen_host(make_inputs(p, 4), tag="varlen_f32_small")


def test_varlen_host_offsets_per_sequence_and_many(tune):
    """The per-sequence launches (forced), and more sequences than one launch
    takes by value (they run per sequence)."""
    p = Problem(1, 3000, 8, 64, 128, 4, 256, "bf16", varlen=True, len_lo=1, len_hi=700, init_states=True)
    tune("varlen_per_sequence", 1)
    check_varlen_host(make_inputs(p, 9), tag="varlen_per_sequence_forced")
    tune("varlen_per_sequence", 0)
    inp = _packed(np.random.default_rng(7).integers(1, 4, 600).tolist() + [500], 2, 64, 1, 43)
    check_varlen_host(inp, tag="varlen_601_sequences")


def test_varlen_host_offsets_full_size():
    check_varlen_host(make_inputs(WORKLOADS["varlen_g8"], 0), tag="varlen_g8")
