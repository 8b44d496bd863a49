"""GPU parity of kf_group_norm against the float64 oracle across shapes that
exercise every path: single-chunk groups, fused multi-chunk groups with the
cross-workgroup exchange (and its recompute fallback), the two-launch paths
for grids that cannot be co-resident and for in-place calls, scalar (non-vectorisable) layouts, every dtype and
affine combination, in-place use, determinism and workspace hygiene.

Tolerances: bf16 / fp16 outputs within 1 unit in the last place of the
oracle rounded once, except where |oracle| < 2^-19: there an absolute error
<= 2^-22 is also accepted (fp32 statistics cannot resolve a bf16 ulp that
small; strict counts are reported).  fp32 outputs: max abs error <= 1e-6."""
import numpy as np
import pytest
import torch

from compare import assert_close, note
from exchange_child import inputs, spawn
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd import workloads as W
from paper_2607_24762_amd.workloads import randn

pytestmark = pytest.mark.gpu
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
FLOOR = (2.0 ** -19, 2.0 ** -22)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


def check(y, ref, dt):
    if dt == "f32":
        r = assert_close(y, ref, "f32")
        print(f"[parity] fp32 group_norm max_abs {r['max_abs']:.3e}", flush=True)
        return
    assert_close(y, ref, dt, floor=FLOOR)


def run(shape, groups, dt, affine="same", eps=1e-6, seed=0, mean=0.3, std=1.5, in_place=False,
        channels_last=False):
    c = shape[1]
    x_cpu = randn(shape, dt, seed=seed, mean=mean, std=std)
    adt = dt if affine == "same" else "f32"
    w_cpu = randn((c,), adt, seed=seed + 1, mean=1.0, std=0.1) if affine in ("same", "f32", "w") else None
    b_cpu = randn((c,), adt, seed=seed + 2, std=0.1) if affine in ("same", "f32", "b") else None
    x = x_cpu.cuda()
    if channels_last:
        x = x.contiguous(memory_format=torch.channels_last)
    w = w_cpu.cuda() if w_cpu is not None else None
    b = b_cpu.cuda() if b_cpu is not None else None
    y = kf355.kf_group_norm(x, groups, w, b, eps, out=x if in_place else None)
    torch.cuda.synchronize()
    variant = kf355.last_variant()
    ref = oracle.group_norm(x_cpu, groups, w_cpu, b_cpu, eps)
    check(y, ref, dt)
    return y, variant


SHAPES = [
    ((2, 8), 4),                 # [N, C]: one element per channel
    ((3, 6, 10), 3),             # [N, C, L]
    ((2, 64, 8, 8), 8),          # small groups, one chunk each
    ((1, 32, 7, 7), 4),          # spatial 49: not whole vectors -> scalar layout
    ((4, 320, 32, 32), 32),      # SD-style 10-channel groups, one chunk
    ((1, 128, 64, 64), 32),      # exactly one full chunk per group
    ((2, 512, 64, 64), 32),      # 4-chunk groups, 256 workgroups
    ((1, 32, 256, 256), 1),      # one 2M-element group: 128 chunks
    ((1, 16, 3, 5, 7), 4),       # 3-D spatial, ragged chunk tail
]


@pytest.mark.parametrize("dt", ["bf16", "f32", "f16"])
@pytest.mark.parametrize("shape,groups", SHAPES, ids=lambda v: str(v))
def test_shape_sweep(shape, groups, dt):
    note(f"group_norm {shape} G={groups} {dt}")
    _, variant = run(shape, groups, dt)
    assert variant.startswith("gn_"), variant


@pytest.mark.parametrize("affine", ["f32", "w", "b", "none"])
def test_affine_variants(affine):
    note(f"group_norm affine={affine}")
    run((2, 64, 32, 32), 16, "bf16", affine=affine)


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("affine", ["same", "f32", "w", "b", "none"])
def test_affine_variants_multi_chunk(affine, dt):
    # 4 chunks per group with the cross-workgroup exchange, where an absent
    # weight or bias reads the identity element of the affine dtype instead
    # of branching: gn_pipe for 16-bit tensors, the fused kernel for fp32.
    note(f"group_norm multi-chunk affine={affine} {dt}")
    _, variant = run((1, 64, 64, 64), 4, dt, affine=affine)
    assert variant == ("gn_fused_vec" if dt == "f32" else "gn_pipe_nv8_r1"), variant


@pytest.mark.parametrize("shape,groups", [
    ((1, 512, 128, 128), 32),    # the SD3.5 VAE block: 16 parts per group
    ((1, 64, 128, 128), 8),      # 8 parts per group, 8 groups
    ((3, 32, 64, 64), 4),        # 12 groups of 2 parts: no per-XCD placement
    ((1, 32, 512, 512), 32),     # one 256K-element channel per group, 16 parts
    ((2, 512, 128, 128), 32),    # 64 groups of 16 parts: one round if resident, else two
], ids=lambda v: str(v))
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_pipe_plans(shape, groups, dt):
    note(f"group_norm gn_pipe {shape} G={groups} {dt}")
    _, variant = run(shape, groups, dt, seed=5)
    assert variant in ("gn_pipe_nv8_r1", "gn_pipe_nv8_r2"), variant


def test_pipe_exact_moments_fallback():
    # Channels whose mean is large against their spread (mean^2 > 63 var over
    # a wave's 4096 values) make the raw-sum moments cancel; those waves
    # recompute them exactly.  Mixed with ordinary channels in one group.
    note("group_norm gn_pipe exact-moment fallback")
    x = randn((1, 64, 64, 64), "bf16", seed=9, mean=0.3, std=1.5)
    x[:, 8:12] = randn((1, 4, 64, 64), "bf16", seed=10, mean=40.0, std=0.25)
    x[:, 40:48] = randn((1, 8, 64, 64), "bf16", seed=11, mean=-300.0, std=2.0)
    w = randn((64,), "bf16", seed=12, mean=1.0, std=0.1)
    b = randn((64,), "bf16", seed=13, std=0.1)
    y = kf355.kf_group_norm(x.cuda(), 4, w.cuda(), b.cuda(), 1e-6)
    torch.cuda.synchronize()
    assert kf355.last_variant() == "gn_pipe_nv8_r1"
    check(y, oracle.group_norm(x, 4, w, b, 1e-6), "bf16")


def test_two_launch_path_for_grids_that_cannot_be_resident():
    # 8 samples x 32 groups x 16 chunks = 4096 workgroups of 4 waves: a CU
    # holds at most 32 waves, so no device of 256 CUs can hold more than 2048
    # of them at once (gn_pipe's workgroups have a fifth wave).  Dense NCHW
    # 16-bit: gn_split's two launches; the general two-kernel form is pinned
    # by the forced plans below.
    note("group_norm split (8,128,256,256)")
    props = torch.cuda.get_device_properties(0)
    assert 4096 > props.multi_processor_count * 32 // 4
    _, variant = run((8, 128, 256, 256), 32, "bf16", seed=4)
    assert variant == "gn_split_nv8", variant


SPLIT_CASES = [
    ((1, 64, 512, 512), 1, "bf16", "same"),    # one 16M-element group: 1024 parts, 16 per lane
    ((1, 32, 512, 512), 2, "bf16", "f32"),     # 256 parts per group, fp32 affine
    ((1, 32, 512, 512), 2, "f16", "none"),     # fp16, no affine
    ((2, 16, 512, 1024), 2, "f16", "same"),    # 256 parts per group, two samples
    ((1, 64, 256, 512), 1, "bf16", "w"),       # 512 parts, weight only
]


@pytest.mark.parametrize("shape,groups,dt,affine", SPLIT_CASES, ids=lambda v: str(v))
def test_split_path_matches_the_oracle(shape, groups, dt, affine):
    # Groups of more than 64 parts even in 32768-element chunks: gn_pipe's
    # one-wave gather cannot take them, gn_split's two launches do (the last
    # arrival of a group folds its parts 2 to 16 per lane, then the lane
    # butterfly).  Parity with the oracle, bit-identical repeats, and the
    # workspace left zero after the status block with no give-up.
    note(f"group_norm split {shape} G={groups} {dt} affine={affine}")
    y, variant = run(shape, groups, dt, affine=affine, seed=21, mean=-0.7, std=2.0)
    assert variant == "gn_split_nv8", variant
    x = randn(shape, dt, seed=21, mean=-0.7, std=2.0).cuda()
    c = shape[1]
    adt = dt if affine == "same" else "f32"
    w = randn((c,), adt, seed=22, mean=1.0, std=0.1).cuda() if affine in ("same", "f32", "w") else None
    b = randn((c,), adt, seed=23, std=0.1).cuda() if affine in ("same", "f32", "b") else None
    ws = torch.zeros(kf355.kf_group_norm_workspace_bytes(x, groups), dtype=torch.uint8, device="cuda")
    y1 = kf355.kf_group_norm(x, groups, w, b, 1e-6, workspace=ws)
    y2 = kf355.kf_group_norm(x, groups, w, b, 1e-6, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    assert torch.equal(y1.view(torch.int16), y.view(torch.int16))
    assert kf355.workspace_give_ups(ws) == 0
    assert int(ws[256:].count_nonzero().item()) == 0


def test_a_call_needs_only_its_layouts_workspace():
    # The size query, blind to layout, covers channels last (270592 bytes for
    # the SD3.5 block: 64 parts per group, one line each); an NCHW call needs
    # only its own layout's 12544 bytes and accepts exactly that, one byte
    # less is KF_ERR_WORKSPACE, and the workspace comes back zero.
    note("group_norm NCHW workspace of its own layout")
    a = inputs("group_norm")
    x, w, b = a["x"].cuda(), a["weight"].cuda(), a["bias"].cuda()
    assert kf355.kf_group_norm_workspace_bytes(x, 32) == 270592
    ws = torch.zeros(12544, dtype=torch.uint8, device="cuda")   # 256 + 32 * 16 * 8 + 32 * 256
    y = kf355.kf_group_norm(x, 32, w, b, a["eps"], workspace=ws)
    torch.cuda.synchronize()
    assert kf355.last_variant() == "gn_pipe_nv8_r1"
    check(y.cpu(), oracle.group_norm(a["x"], 32, a["weight"], a["bias"], a["eps"]), "bf16")
    assert int(ws[256:].count_nonzero().item()) == 0
    with pytest.raises(kf355.KfError) as e:
        kf355.kf_group_norm(x, 32, w, b, a["eps"], workspace=ws[:12543])
    assert e.value.status == 6


def test_split_recompute_is_bit_identical(tmp_path):
    # KF355_GN_SPLIT_RECOMPUTE=1 makes each group's last arrival recompute
    # every part from x, as it does when a published part stays unseen: the
    # same bits, one give-up per group, the workspace zero again.
    note("group_norm split with the recompute path forced")
    a = spawn(tmp_path, ["group_norm_split"])
    b = spawn(tmp_path, ["group_norm_split"], KF355_GN_SPLIT_RECOMPUTE="1")
    assert str(a["variant0"]) == str(b["variant0"]) == "gn_split_nv8"
    assert int(a["give_ups"]) == 0 and int(b["give_ups"]) == inputs("group_norm_split")["groups"]
    assert int(a["rest"]) == 0 and int(b["rest"]) == 0
    assert np.array_equal(a["bits0"], b["bits0"])
    i = inputs("group_norm_split")
    check(_as_tensor(b["bits0"]), oracle.group_norm(i["x"], i["groups"], i["weight"], i["bias"], i["eps"]), "bf16")


def test_in_place():
    # In place: gn_pipe's chunks of a group would be overwritten while its
    # recompute fallback might still read them, so multi-chunk groups take
    # gn_split (whose second launch reads each chunk before writing it) or,
    # where gn_split does not apply (spatial size not a multiple of 2048),
    # the general two-kernel form.
    note("group_norm in place")
    _, variant = run((1, 512, 64, 64), 32, "bf16", in_place=True, seed=6)   # 4 chunks per group
    assert variant == "gn_split_nv8", variant
    _, variant = run((1, 32, 64, 64), 4, "f16", in_place=True, seed=9)     # 2 chunks per group, the fewest
    assert variant == "gn_split_nv8", variant
    _, variant = run((1, 256, 48, 48), 32, "bf16", in_place=True, seed=7)   # 2 chunks, spatial 2304
    assert variant.startswith("gn_two_pass"), variant
    _, variant = run((2, 64, 8, 8), 8, "bf16", in_place=True, seed=8)
    assert variant.startswith("gn_fused"), variant  # one chunk per group: no exchange


def test_constant_groups_give_bias():
    note("group_norm constant groups")
    x = torch.full((1, 64, 16, 16), 0.75, dtype=torch.bfloat16, device="cuda")
    b = randn((64,), "bf16", seed=2).cuda()
    y = kf355.kf_group_norm(x, 8, None, b, 1e-6)
    torch.cuda.synchronize()
    assert torch.equal(y, b.view(1, 64, 1, 1).expand_as(y))


def test_repeat_calls_bitwise_identical_and_workspace_clean():
    note("group_norm determinism x1000 (1,512,128,128)")
    x = randn((1, 512, 128, 128), "bf16", seed=3, mean=0.3, std=1.5).cuda()
    w = randn((512,), "bf16", seed=4, mean=1.0, std=0.1).cuda()
    b = randn((512,), "bf16", seed=5, std=0.1).cuda()
    ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    ref = kf355.kf_group_norm(x, 32, w, b, 1e-6, workspace=ws)
    y = torch.empty_like(ref)
    bad = torch.zeros((), dtype=torch.int64, device="cuda")
    for _ in range(1000):
        kf355.kf_group_norm(x, 32, w, b, 1e-6, out=y, workspace=ws)
        bad += (y.view(torch.int16) != ref.view(torch.int16)).sum()
    torch.cuda.synchronize()
    assert int(bad.item()) == 0
    # Every call empties its partial slots and counters, and no wait gave
    # up: the whole workspace is zero again.
    assert int(ws.count_nonzero().item()) == 0


def test_wait_timeout_recompute_is_bitwise_identical(tmp_path):
    # A child process with KF355_GN_WAIT_TICKS=0 makes every workgroup that
    # does not find its whole group published on the first poll recompute the
    # group's statistics itself; the output must equal the normal path's bit
    # for bit, the give-up count must be non-zero and everything after the
    # status block left zero.
    note("group_norm forced-timeout recompute")
    w = W.groupnorm_vae_bf16()
    y = kf355.kf_group_norm(w["x"].cuda(), 32, w["weight"].cuda(), w["bias"].cuda(), w["eps"])
    torch.cuda.synchronize()
    got = spawn(tmp_path, ["group_norm"], KF355_GN_WAIT_TICKS="0")
    assert str(got["variant0"]) == "gn_pipe_nv8_r1"
    assert int(got["give_ups"]) >= 1
    assert int(got["rest"]) == 0
    assert np.array_equal(got["bits0"], y.view(torch.int16).cpu().numpy())


def test_fused_kernel_wait_timeout_recompute_is_bitwise_identical(tmp_path):
    # The same for the fused kernel gn_pipe replaced on 16-bit NCHW tensors
    # (still used for fp32, channels last and shapes outside gn_pipe):
    # KF355_GN_MODE=fused selects it, once with the normal wait and once with
    # every wait given up at once.
    note("group_norm fused-kernel forced-timeout recompute")
    a = spawn(tmp_path, ["group_norm"], KF355_GN_MODE="fused")
    b = spawn(tmp_path, ["group_norm"], KF355_GN_MODE="fused", KF355_GN_WAIT_TICKS="0")
    assert str(a["variant0"]) == "gn_fused_vec" and str(b["variant0"]) == "gn_fused_vec"
    assert int(a["give_ups"]) == 0 and int(b["give_ups"]) >= 1
    assert int(a["rest"]) == 0 and int(b["rest"]) == 0
    assert np.array_equal(a["bits0"], b["bits0"])
    w = W.groupnorm_vae_bf16()
    ref = oracle.group_norm(w["x"], 32, w["weight"], w["bias"], w["eps"])
    check(_as_tensor(a["bits0"]), ref, "bf16")


@pytest.mark.parametrize("parts,want", [(1, "gn_pipe_nv8_r1"), (2, "gn_pipe_nv4_r1"), (4, "gn_pipe_nv2_r1")])
def test_forced_parts_per_group_deterministic(tmp_path, parts, want):
    # KF355_GN_PARTS forces the number of workgroups per group (1, 2 and the
    # most the smallest chunk gives for this shape): each setting matches the
    # oracle, two calls give identical bits, no wait gives up and the
    # workspace is left zero.
    note(f"group_norm forced parts per group = {parts}")
    got = spawn(tmp_path, ["group_norm_parts", "group_norm_parts"], KF355_GN_PARTS=str(parts))
    assert str(got["variant0"]) == want and str(got["variant1"]) == want
    assert int(got["give_ups"]) == 0 and int(got["rest"]) == 0
    assert np.array_equal(got["bits0"], got["bits1"])
    a = inputs("group_norm_parts")
    ref = oracle.group_norm(a["x"], a["groups"], a["weight"], a["bias"], a["eps"])
    check(_as_tensor(got["bits0"]), ref, "bf16")


@pytest.mark.parametrize("env,want", [
    ({"KF355_GN_PARTS": "64"}, ("gn_pipe_nv2_r1", "gn_pipe_nv2_r2")),  # 4096-element chunks, the most parts
    ({"KF355_GN_PARTS": "8"}, ("gn_pipe_nv16_r1",)),                  # 32768-element chunks: two channels each
    ({"KF355_GN_ROUNDS": "2"}, ("gn_pipe_nv8_r2",)),                  # two rounds of 16 groups
    ({"KF355_GN_MODE": "two_pass"}, ("gn_two_pass_vec",)),            # the general two-kernel form
], ids=["parts64", "parts8", "rounds2", "two_pass"])
def test_pipe_forced_plans_on_the_vae_block(tmp_path, env, want):
    # The SD3.5 VAE block under plans the default does not pick: each matches
    # the oracle, repeats bit for bit, gives up no wait and leaves the
    # workspace zero.
    note(f"group_norm gn_pipe forced plan {env}")
    got = spawn(tmp_path, ["group_norm", "group_norm"], **env)
    assert str(got["variant0"]) in want, got["variant0"]
    assert int(got["give_ups"]) == 0 and int(got["rest"]) == 0
    assert np.array_equal(got["bits0"], got["bits1"])
    a = inputs("group_norm")
    check(_as_tensor(got["bits0"]), oracle.group_norm(a["x"], a["groups"], a["weight"], a["bias"], a["eps"]), "bf16")


def test_staggered_issue_changes_no_bit(tmp_path):
    # On the SD3.5 VAE block (512 workgroups, two per CU) the second half of
    # gn_pipe's grid issues its loads later; with that wait off every output
    # bit is the same, and neither run gives up a wait.
    note("group_norm gn_pipe with and without the staggered issue")
    a = spawn(tmp_path, ["group_norm"])
    b = spawn(tmp_path, ["group_norm"], KF355_GN_STAGGER_TICKS="0")
    assert str(a["variant0"]) == str(b["variant0"]) == "gn_pipe_nv8_r1"
    assert int(a["give_ups"]) == 0 and int(b["give_ups"]) == 0
    assert int(a["rest"]) == 0 and int(b["rest"]) == 0
    assert np.array_equal(a["bits0"], b["bits0"])


def _oracle_of(op):
    a = inputs(op)
    if op == "softmax_split":
        return oracle.softmax(a["x"], -1), "f32"
    return oracle.group_norm(a["x"], a["groups"], a["weight"], a["bias"], a["eps"]), "bf16"


def _as_tensor(bits):
    t = torch.from_numpy(bits)
    return t.view(torch.bfloat16) if t.dtype == torch.int16 else t.view(torch.float32)


@pytest.mark.parametrize("env,ops", [
    ({"KF355_SM_WAIT_TICKS": "0"}, ["softmax_split", "group_norm", "group_norm_small"]),
    ({"KF355_GN_WAIT_TICKS": "0"}, ["group_norm_small", "softmax_split", "group_norm"]),
    ({"KF355_GN_WAIT_TICKS": "0"}, ["group_norm", "group_norm_small", "group_norm"]),
], ids=["split-gave-up", "small-gave-up", "large-gave-up"])
def test_give_up_count_never_corrupts_later_calls(tmp_path, env, ops):
    # A call whose workgroups gave up leaves a non-zero give-up count in the
    # workspace; later calls of other shapes and of the other operator on the
    # same workspace must still match the oracle, and leave every byte after
    # the status block zero.
    note(f"exchange workspace reuse after give-ups {env} {ops}")
    got = spawn(tmp_path, ops, **env)
    assert int(got["give_ups"]) >= 1
    assert int(got["rest"]) == 0
    for i, op in enumerate(ops):
        ref, fmt = _oracle_of(op)
        assert_close(_as_tensor(got[f"bits{i}"]), ref, fmt, **({"floor": FLOOR} if fmt == "bf16" else {}))


def test_concurrent_calls_on_two_streams():
    note("group_norm two streams")
    w = W.groupnorm_vae_bf16()
    x, g, b = w["x"].cuda(), w["weight"].cuda(), w["bias"].cuda()
    ref = kf355.kf_group_norm(x, 32, g, b, w["eps"])
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for _ in range(20):
        with torch.cuda.stream(s1):
            outs.append(kf355.kf_group_norm(x, 32, g, b, w["eps"]))
        with torch.cuda.stream(s2):
            outs.append(kf355.kf_group_norm(x, 32, g, b, w["eps"]))
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int16), ref.view(torch.int16))


@pytest.mark.parametrize("mode_shape", [((1, 512, 128, 128), 32), ((2, 64, 8, 8), 8)])
def test_paths_share_one_workspace(mode_shape):
    # Alternating shapes (different chunk counts) through one workspace:
    # each call must find it empty.
    note(f"group_norm shared workspace {mode_shape}")
    ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    for shape, groups in [mode_shape, ((1, 128, 64, 64), 32), mode_shape]:
        x_cpu = randn(shape, "bf16", seed=7, mean=0.3, std=1.5)
        y = kf355.kf_group_norm(x_cpu.cuda(), groups, None, None, 1e-6, workspace=ws)
        torch.cuda.synchronize()
        assert_close(y, oracle.group_norm(x_cpu, groups, None, None, 1e-6), "bf16", floor=FLOOR)
    assert int(ws.count_nonzero().item()) == 0


CHANNELS_LAST = [
    ((1, 512, 128, 128), 32),    # the SD3.5 VAE block, channels last: 16-chunk groups
    ((2, 64, 15, 17), 8),        # 8-channel groups, ragged pixel count
    ((2, 96, 9, 7), 96),         # one channel per group: scalar layout
    ((1, 24, 64, 64), 2),        # 12-channel groups: scalar layout, 3 chunks
    ((3, 256, 10, 5), 1),        # one group of every channel
    ((2, 32, 60, 50), 2),        # 16-channel groups, 3 chunks
    ((2, 64, 48, 45), 8),        # 8-channel groups, 2 chunks per group, the last one ragged
    ((2, 128, 36, 23), 4),       # 32-channel groups, 2 chunks per group, the last one ragged
]



@pytest.mark.parametrize("dt", ["bf16", "f32", "f16"])
@pytest.mark.parametrize("shape,groups", CHANNELS_LAST, ids=lambda v: str(v))
def test_channels_last(shape, groups, dt):
    note(f"group_norm channels last {shape} G={groups} {dt}")
    y, variant = run(shape, groups, dt, channels_last=True)
    assert y.is_contiguous(memory_format=torch.channels_last)
    cpg = shape[1] // groups
    if dt != "f32" and cl_parts(shape, groups):
        assert variant == f"gn_pipe_cl_cpg{cpg}", variant
        return
    assert variant.startswith("gn_nhwc_"), variant
    vec = 4 if dt == "f32" else 8
    assert ("_vec" in variant) == (cpg % vec == 0 and (256 * vec) % cpg == 0), variant


def cl_parts(shape, groups):
    """Parts per group of the channels-last tile kernel (16-bit tensors):
    tiles of 64 channels x 256 pixels, c a multiple of 64, 8 to 64 channels
    per group, 2 to 64 parts (a power of two); 0 where it does not apply."""
    c, hw = shape[1], int(np.prod(shape[2:]))
    cpg = c // groups
    if c % 64 or cpg not in (8, 16, 32, 64) or hw % 256:
        return 0
    parts = hw // 256
    return parts if 2 <= parts <= 64 and parts & (parts - 1) == 0 else 0


CL_TILES = [
    ((1, 512, 128, 128), 32),    # the SD3.5 VAE block: 16 channels per group, 64 parts, 8 tile columns
    ((2, 128, 16, 32), 4),       # 32 channels per group, 2 parts, two samples
    ((3, 256, 32, 64), 16),      # 16 channels per group, 8 parts, 12 tile columns
    ((1, 256, 64, 64), 32),      # 8 channels per group, 16 parts
    ((2, 512, 32, 32), 8),       # 64 channels per group, 4 parts, 16 tile columns
    ((1, 128, 128, 128), 4),     # 32 channels per group, 64 parts
    ((1, 512, 64, 128), 64),     # 8 channels per group, 64 groups, 32 parts
    ((2, 64, 32, 32), 8),        # 64 channels: 8 per group, 4 parts, one tile column per sample
    ((1, 192, 64, 64), 3),       # 64 channels per group, 16 parts, 3 tile columns (not a multiple of 8)
    ((1, 1024, 32, 32), 32),     # 32 channels per group, 4 parts, 16 tile columns (two per XCD)
    ((2, 384, 16, 32), 12),      # 32 channels per group, 2 parts, 12 tile columns
    ((1, 640, 32, 32), 80),      # 8 channels per group, 4 parts, 10 tile columns
    ((1, 64, 128, 128), 4),      # 16 channels per group, 64 parts, one tile column
]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("affine", ["same", "f32", "none"])
@pytest.mark.parametrize("shape,groups", CL_TILES, ids=lambda v: str(v))
def test_channels_last_tiles(shape, groups, affine, dt):
    """The channels-last tile kernel at every group width, 2 to 64 parts
    and 1 to 16 tile columns, against the oracle; two calls give identical
    bits."""
    assert cl_parts(shape, groups)
    note(f"group_norm channels last tiles {shape} G={groups} affine={affine} {dt}")
    y, variant = run(shape, groups, dt, affine=affine, channels_last=True, seed=len(shape) + groups)
    assert variant == f"gn_pipe_cl_cpg{shape[1] // groups}", variant
    y2, _ = run(shape, groups, dt, affine=affine, channels_last=True, seed=len(shape) + groups)
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("shape,groups", [((1, 256, 32, 64), 16), ((1, 192, 32, 32), 3)], ids=["cpg16", "cpg64"])
def test_channels_last_large_mean(shape, groups):
    # A mean large against the spread takes the exact M2 path of the moments.
    note(f"group_norm channels last {shape}, mean 40 std 0.05")
    run(shape, groups, "bf16", channels_last=True, mean=40.0, std=0.05)


@pytest.mark.parametrize("affine", ["none", "w", "b", "f32"])
def test_channels_last_affine_and_in_place(affine):
    note(f"group_norm channels last affine={affine}")
    run((2, 64, 32, 32), 4, "bf16", affine=affine, channels_last=True)
    _, variant = run((1, 128, 64, 64), 8, "bf16", affine=affine, channels_last=True, in_place=True)
    assert variant == "gn_nhwc_two_pass_vec", variant     # multi-chunk in place: two kernels


def test_channels_last_matches_nchw_statistics():
    # The same logical tensor in both layouts normalises to the same values
    # within the tolerance (the moment merges visit elements in different orders).
    note("group_norm channels last vs NCHW")
    w = W.groupnorm_vae_bf16()
    x = w["x"].cuda()
    a = kf355.kf_group_norm(x, 32, w["weight"].cuda(), w["bias"].cuda(), w["eps"])
    b = kf355.kf_group_norm(x.contiguous(memory_format=torch.channels_last), 32, w["weight"].cuda(),
                            w["bias"].cuda(), w["eps"])
    torch.cuda.synchronize()
    assert b.is_contiguous(memory_format=torch.channels_last)
    ref = oracle.group_norm(w["x"], 32, w["weight"], w["bias"], w["eps"])
    check(a, ref, "bf16")
    check(b, ref, "bf16")


@pytest.mark.parametrize("op,variant", [("group_norm_nhwc", "gn_pipe_cl_cpg16"),
                                        ("group_norm_tiles_small", "gn_pipe_cl_cpg64")])
def test_channels_last_gave_up_waiting_recomputes_bit_identically(tmp_path, op, variant):
    # With no wait at all every workgroup recomputes the parts it lacks
    # from the tensor; the output must not change by a bit and the exchange
    # must be left zero.
    note(f"group_norm channels last forced recompute {op} (child process)")
    a = inputs(op)
    x = a["x"].cuda().contiguous(memory_format=torch.channels_last)
    y = kf355.kf_group_norm(x, a["groups"], a["weight"].cuda(), a["bias"].cuda(), a["eps"])
    torch.cuda.synchronize()
    assert kf355.last_variant() == variant
    got = spawn(tmp_path, [op, op], KF355_GN_WAIT_TICKS="0")
    assert str(got["variant0"]) == variant and str(got["variant1"]) == variant
    assert int(got["give_ups"]) >= 1 and int(got["rest"]) == 0
    bits = y.contiguous().view(torch.int16).cpu().numpy()
    assert np.array_equal(got["bits0"], bits) and np.array_equal(got["bits1"], bits)
    ref = oracle.group_norm(a["x"], a["groups"], a["weight"], a["bias"], a["eps"])
    check(y, ref, "bf16")