"""The library's choice of kernels per shape, through iabn_plan (host only,
no GPU): which path runs, the block and register depth of the
channel-resident kernels, what waits in LDS, strip addressing, access
width and the XCD order.  These are the decisions the measurements behind
the kernels settled; a change to any of them shows up here first.
"""

import pytest
import torch

import paper_1712_02616_amd as iabn

F32, F16, BF16 = torch.float32, torch.float16, torch.bfloat16


def plan(op, dtype, N, C, HW):
    return iabn.iabn_plan(op, dtype, N, C, HW)


def fused(p, T, R, lds=0, strips=None, access=16, xcd=0, blocks=None, cpb=1):
    """T: threads per channel; cpb: channels per block."""
    assert p["channel_resident"] == 1, p
    assert p["channels_per_block"] == cpb, p
    assert (p["threads"], p["reg_accesses"], p["lds_accesses"]) == (T * cpb, R, lds), p
    assert p["access_bytes"] == access and p["xcd_order"] == xcd, p
    if strips is not None:
        assert p["strips"] == strips, p
    if blocks is not None:
        assert p["blocks"] == blocks, p


def streaming(p, access=16, xcd=0, blocks=None):
    assert p["channel_resident"] == 0 and p["threads"] == 256, p
    assert p["channels_per_block"] == 0, p
    assert p["reg_accesses"] == p["lds_accesses"] == p["strips"] == 0, p
    assert p["access_bytes"] == access and p["xcd_order"] == xcd, p
    if blocks is not None:
        assert p["blocks"] == blocks, p


@pytest.mark.parametrize("op", ["forward_train", "backward"])
def test_backbone_sweep_layers(op):
    """The four layer shapes of the benchmark's sweep (fp16, N = 8)."""
    bwd = op == "backward"
    # C = 256 at 128x128: 16 strips of 1024 accesses; the backward keeps 11 in
    # registers and 4 in LDS.
    fused(plan(op, F16, 8, 256, 128 * 128), 1024, 11 if bwd else 16, lds=4 if bwd else 0,
          strips=1, blocks=256)
    for C in (512, 1024, 2048):
        # Two channels per block: the forward from 1024 to 2047 channels, the
        # backward for 512 and 1024 (whole rounds of one block per CU).
        cpb = 2 if (C in (512, 1024) if bwd else C == 1024) else 1
        fused(plan(op, F16, 8, C, 64 * 64), 256, 16, strips=1, blocks=C // cpb, cpb=cpb)


def test_two_channel_forward_blocks():
    """The forward's (256, 16) rung on rows of whole strips: two adjacent
    channels per block for 1024-2047 (even) channels, every forward mode;
    one per block outside that range, for odd channel counts, for rows that
    take the general mapping, and in the backward."""
    for op in ("forward_train", "std_forward", "ckpt_forward"):
        fused(plan(op, F16, 8, 1024, 64 * 64), 256, 16, strips=1, blocks=512, cpb=2)
        fused(plan(op, F16, 8, 1536, 64 * 64), 256, 16, strips=1, blocks=768, cpb=2)
        fused(plan(op, F16, 8, 2046, 64 * 64), 256, 16, strips=1, blocks=1023, cpb=2)
    fused(plan("forward_train", F16, 8, 1022, 64 * 64), 256, 16, strips=1, blocks=1022)
    fused(plan("forward_train", F16, 8, 1025, 64 * 64), 256, 16, strips=1, blocks=1025)
    fused(plan("forward_train", F32, 8, 1024, 32 * 64), 256, 16, strips=1, blocks=512, cpb=2)
    # Rows of 32x32 fp16 (128 accesses) hold no 256-wide strip: general mapping.
    fused(plan("forward_train", F16, 32, 1024, 32 * 32), 256, 16, strips=0, blocks=1024)



def test_multi_channel_backward_blocks():
    """Every backward (InPlace-ABN I and II, the standard block, the
    checkpointing) takes several adjacent channels per (256, 16) block where
    the launch is then one round of one block per CU (512 channels: two per
    block, 768: three, on 256 CUs) and two per block for 1024 channels."""
    fused(plan("backward", F16, 8, 512, 64 * 64), 256, 16, strips=1, blocks=256, cpb=2)
    fused(plan("backward", F16, 8, 768, 64 * 64), 256, 16, strips=1, blocks=256, cpb=3)
    fused(plan("backward", F16, 8, 1024, 64 * 64), 256, 16, strips=1, blocks=512, cpb=2)
    fused(plan("backward", F32, 8, 512, 32 * 64), 256, 16, strips=1, blocks=256, cpb=2)
    for C in (256, 1280, 1536, 2048):
        fused(plan("backward", F16, 8, C, 64 * 64), 256, 16, strips=1, blocks=C)
    for op in ("std_backward", "ckpt_backward"):
        fused(plan(op, F16, 8, 512, 64 * 64), 256, 16, strips=1, blocks=256, cpb=2)
        fused(plan(op, F16, 8, 768, 64 * 64), 256, 16, strips=1, blocks=256, cpb=3)
        fused(plan(op, F16, 8, 2048, 64 * 64), 256, 16, strips=1, blocks=2048)
    # Rows that take the general mapping keep one channel per block.
    fused(plan("backward", F16, 32, 512, 32 * 32), 256, 16, strips=0, blocks=512)


def test_parity_workloads():
    # ResNet layer, fp32: 25088 accesses per channel, the last rung with LDS.
    fused(plan("forward_train", F32, 32, 256, 56 * 56), 1024, 16, lds=9, strips=0)
    fused(plan("backward", F32, 32, 256, 56 * 56), 1024, 11, lds=4, strips=0)
    # Segmentation crop: 18432 accesses, two strips past the forward's registers.
    fused(plan("forward_train", F16, 4, 256, 192 * 192), 1024, 16, lds=2, strips=0)
    # Wide layer: 1568 accesses per channel, rows of 1568 bytes (not whole
    # lines); 2048 channels: the forward takes one wave per channel.
    fused(plan("forward_train", BF16, 16, 2048, 28 * 28), 64, 32, strips=0, xcd=1, blocks=2048)
    fused(plan("backward", BF16, 16, 2048, 28 * 28), 256, 8, strips=0, xcd=1, blocks=2048)
    # Tiny layer: streaming.
    streaming(plan("forward_train", F32, 2, 16, 8 * 8))


def test_few_channel_rule():
    # Forward from 64 channels, backward from 96, while a channel fits.
    fused(plan("forward_train", F16, 32, 64, 56 * 56), 1024, 16)
    streaming(plan("backward", F16, 32, 64, 56 * 56))
    fused(plan("backward", F16, 32, 96, 56 * 56), 1024, 11, lds=2)
    streaming(plan("forward_train", F16, 32, 63, 56 * 56))
    # Up to 16K accesses below 128 channels, 32K from 128.
    streaming(plan("forward_train", F16, 8, 96, 256 * 256 // 2))
    fused(plan("forward_train", F32, 32, 128, 56 * 56), 1024, 16, lds=9)
    streaming(plan("forward_train", F16, 8, 128, 36864))
    # A stem-like layer (64 channels of 256x256) stays on the streaming kernels.
    streaming(plan("forward_train", F16, 8, 64, 256 * 256), blocks=64 * 8)
    streaming(plan("backward", F16, 8, 64, 256 * 256), blocks=64 * 8)


def test_rungs():
    # 1025-2048 accesses: (256, 8) on the 16-byte path.
    fused(plan("forward_train", F16, 8, 300, 2048), 256, 8, strips=1)
    fused(plan("backward", F16, 8, 300, 2048), 256, 8, strips=1)
    # Narrow rows with at most one channel per CU: (512, 4); with more: (256, 8).
    fused(plan("backward", F16, 32, 200, 14 * 14), 512, 4, access=8, xcd=1)
    fused(plan("backward", F16, 32, 1024, 14 * 14), 256, 8, access=8, xcd=1)
    fused(plan("forward_train", F16, 32, 1024, 7 * 7), 256, 8, access=2, xcd=1)
    fused(plan("forward_train", F16, 32, 2048, 7 * 7), 64, 32, access=2, xcd=1)


def test_one_wave_rung():
    """From 2048 channels (two per SIMD) the forward's 1025-2048-access
    channels take one wave each, on every access width; the backward keeps
    (256, 8)."""
    fused(plan("forward_train", F16, 16, 2047, 28 * 28), 256, 8, xcd=1)
    fused(plan("forward_train", F16, 16, 2048, 28 * 28), 64, 32, xcd=1)
    fused(plan("forward_train", F32, 8, 2048, 28 * 28), 64, 32, xcd=1)
    fused(plan("forward_train", F16, 2, 2048, 8192), 64, 32, strips=1)
    fused(plan("std_forward", F16, 16, 4096, 28 * 28), 64, 32, xcd=1)
    fused(plan("ckpt_forward", F16, 16, 4096, 28 * 28), 64, 32, xcd=1)
    fused(plan("forward_train", F16, 32, 2048, 14 * 14), 64, 32, access=8, xcd=1)
    fused(plan("backward", F16, 32, 2048, 14 * 14), 256, 8, access=8, xcd=1)
    fused(plan("std_backward", F16, 16, 2048, 28 * 28), 256, 8, xcd=1)
    # Other rungs are unchanged.
    fused(plan("forward_train", F16, 8, 2048, 64 * 64), 256, 16, strips=1)
    fused(plan("forward_train", F16, 8, 2048, 32 * 32), 256, 4, strips=0)


def test_comparison_blocks():
    # The standard block keeps three tensors in the backward: 3 per tensor in LDS.
    fused(plan("std_backward", F16, 8, 256, 128 * 128), 1024, 11, lds=3, strips=1)
    fused(plan("ckpt_backward", F16, 8, 256, 128 * 128), 1024, 11, lds=4, strips=1)
    fused(plan("std_forward", F16, 8, 1024, 64 * 64), 256, 16, strips=1, cpb=2)
    fused(plan("ckpt_forward", F16, 8, 1024, 64 * 64), 256, 16, strips=1, cpb=2)
    # Narrow rows: the comparison blocks take the streaming kernels.
    streaming(plan("std_forward", F16, 32, 2048, 7 * 7), access=2, xcd=1)
    streaming(plan("ckpt_backward", F16, 32, 2048, 7 * 7), access=2, xcd=1)


def test_always_streaming_entry_points():
    for op in ("forward_eval", "ckpt_recompute"):
        streaming(plan(op, F16, 8, 1024, 64 * 64), blocks=1024)
        streaming(plan(op, F16, 32, 2048, 7 * 7), access=2, xcd=1)
        # Inference accepts a single value per channel (4-byte rows: XCD order).
        streaming(plan(op, F32, 1, 4, 1), access=4, xcd=1)
    # Below 256 channels the inference forward cuts channels into slices for
    # about 8192 blocks (slices of at least 4096 values); the recomputation
    # and the training passes keep about 512.
    streaming(plan("forward_eval", F16, 8, 64, 256 * 256), blocks=8192)
    streaming(plan("forward_eval", F16, 8, 128, 128 * 128), blocks=4096)
    streaming(plan("forward_eval", F16, 8, 256, 128 * 128), blocks=512)
    streaming(plan("ckpt_recompute", F16, 8, 64, 256 * 256), blocks=512)
    streaming(plan("forward_train", F16, 8, 64, 256 * 256), blocks=512)


def test_access_width_and_xcd_order():
    # The widest access that divides a row; XCD order exactly when a row's
    # bytes are not a multiple of 128.
    assert plan("forward_eval", F16, 4, 8, 64)["access_bytes"] == 16     # 128-byte rows
    assert plan("forward_eval", F16, 4, 8, 64)["xcd_order"] == 0
    assert plan("forward_eval", F16, 4, 8, 68)["access_bytes"] == 8      # 136-byte rows
    assert plan("forward_eval", F16, 4, 8, 68)["xcd_order"] == 1
    assert plan("forward_eval", F32, 4, 8, 3)["access_bytes"] == 4
    assert plan("forward_eval", BF16, 4, 8, 3)["access_bytes"] == 2
    assert plan("forward_eval", F32, 4, 8, 96)["xcd_order"] == 0        # 384-byte rows


def test_empty_and_invalid():
    for shape in ((8, 0, 64), (0, 8, 64)):
        assert all(v == 0 for v in plan("forward_eval", F16, *shape).values())
    assert all(v == 0 for v in plan("forward_train", F16, 8, 0, 64).values())
    with pytest.raises(iabn.IabnError) as e:
        plan("forward_train", F16, 1, 4, 1)  # one value per channel in training
    assert e.value.status == 2
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_plan(8, F16, 2, 4, 4)
    assert e.value.status == 3
    with pytest.raises(iabn.IabnError) as e:
        iabn.iabn_plan(0, 7, 2, 4, 4)
    assert e.value.status == 4
    lib = iabn.load()
    assert lib.iabn_plan(0, 1, 2, 4, 4, None) == 1


def test_forward_streaming_partials_fit_the_static_scratch():
    """The training forward takes the streaming kernels (the only ones with a
    scratch buffer) only below 256 channels, where a call's partials never
    exceed 96 KiB: iabn_forward_train_noalloc's 128 KiB scratch holds every
    shape."""
    for C in (256, 300, 1024, 8192, 1 << 20):
        for N, HW in ((1, 2), (8, 4096), (2, 1 << 20)):
            if C * N * HW <= 1 << 46:
                p = iabn.iabn_plan("forward_train", torch.float16, N, C, HW)
                assert p["channel_resident"] == 1, (N, C, HW)
    worst = 0
    for C in range(1, 256):
        for N, HW in ((1, 2), (2, 4096), (8, 65536), (64, 1 << 20)):
            worst = max(worst, iabn.iabn_workspace_size(N, C, HW, torch.float16))
    assert worst <= 96 * 1024, worst
    assert worst == 765 * 4 * 32  # C = 255: 3 slices per channel, 4 partials of 32 bytes each


def test_narrower_accesses_change_the_plan():
    """iabn_plan describes 16-byte-aligned tensors.  A tensor that is not
    (say 8 bytes off) takes the accesses a row that only 8-byte accesses
    divide takes, and that changes the plan, not only its access width: the
    standard block leaves the channel-resident kernels, InPlace-ABN's forward
    takes another rung.  (8, 1024, 4100) fp16 has such rows; the aligned
    neighbour (8, 1024, 4096) does not."""
    fused(plan("std_forward", F16, 8, 1024, 4096), 256, 16, strips=1, cpb=2)
    streaming(plan("std_forward", F16, 8, 1024, 4100), access=8, xcd=1)
    streaming(plan("std_backward", F16, 8, 1024, 4100), access=8, xcd=1)
    fused(plan("forward_train", F16, 8, 1024, 4096), 256, 16, strips=1, cpb=2)
    fused(plan("forward_train", F16, 8, 1024, 4100), 1024, 16, lds=0, access=8, xcd=1)
