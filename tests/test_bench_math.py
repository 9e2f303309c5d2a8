"""The benchmark's counting rules (no GPU): flops and algorithmic HBM bytes
per row, pinned to values worked out by hand from the definitions.

Flops count real dimensions only: the forward is 2 sum fan_in fan_out per
row; the training step adds the backward without the first layer's input
delta and the weight gradients (as many flops as the forward).  Bytes per
row of the three-kernel training step: 4 in + 4 out + 8 d W + 6 OP (OP =
out rounded up to 16), plus the derivative source of the hidden layers:
ReLU masks 2 16 d, sigmoid activations re-read 2 d W, sine cos written and
read 4 d W, linear nothing."""
import bench


def test_flops_per_row_sweep_shapes():
    # (width, inference, training) for in = width, out 16, 4 hidden layers
    for w, inf, train in [(16, 2560, 7168), (32, 9216, 25600), (64, 34816, 96256),
                          (128, 135168, 372736)]:
        assert bench.flops_per_row(w, 4, w, 16) == (inf, train)


def test_flops_per_row_small_cases():
    # depth 0: one in x out matrix, no backward product at all
    assert bench.flops_per_row(64, 0, 40, 12) == (2 * 480, 4 * 480)
    # depth 16, in/out 128: 17 matrices of 128 x 128
    assert bench.flops_per_row(128, 16, 128, 128) == (557056, 557056 * 3 - 2 * 16384)


def test_training_bytes_per_row():
    base = lambda w, d, i, o: 4 * i + 4 * o + 8 * d * w + 6 * ((o + 15) // 16 * 16)
    assert bench.train_bytes_per_row(128, 4, 128, 16, "relu", fused=False) == 4896
    assert bench.train_bytes_per_row(16, 4, 16, 16, "relu", fused=False) == 864
    # the blueprint's three-kernel count, ReLU derivative read from the activations
    assert bench.train_bytes_per_row(128, 4, 128, 16, "relu", fused=False, masks=False) == 5792
    assert bench.train_bytes_per_row(128, 4, 128, 16, "linear") == base(128, 4, 128, 16) == 4768
    assert bench.train_bytes_per_row(128, 4, 128, 16, "sigmoid") == 4768 + 2 * 4 * 128
    assert bench.train_bytes_per_row(128, 4, 128, 16, "sine") == 4768 + 4 * 4 * 128
    # out 3 pads to one 16-column strip for the output delta
    assert bench.train_bytes_per_row(64, 2, 64, 3, "relu", fused=False) == \
        base(64, 2, 64, 3) + 2 * 16 * 2


def test_fused_training_bytes_per_row():
    """Fused plan: 4 in + 4 out + 4 d W + 4 OP, plus at width 128 the ReLU
    masks written and read (2 16 d), or for sine the cos stash (4 d W): no
    hidden delta is written or read."""
    fused = lambda w, d, i, o: 4 * i + 4 * o + 4 * d * w + 4 * ((o + 15) // 16 * 16)
    assert bench.fused_backward(128, 4, 128, 16, "relu")
    # width 128: the ReLU masks written and read (2 16 d)
    assert bench.train_bytes_per_row(128, 4, 128, 16, "relu") == fused(128, 4, 128, 16) + 128 == 2816
    # widths up to 64: relu' from the activations, no masks
    assert bench.train_bytes_per_row(16, 4, 16, 16, "relu", fused=True) == fused(16, 4, 16, 16) == 448
    assert bench.train_bytes_per_row(64, 2, 64, 3, "relu", fused=True) == fused(64, 2, 64, 3)
    assert bench.train_bytes_per_row(64, 2, 64, 3, "sigmoid", fused=True) == fused(64, 2, 64, 3)
    # sine: the cos stash written and read again
    hid = 4 * 64 * 2
    assert bench.train_bytes_per_row(64, 4, 3, 1, "sine", fused=True) == fused(64, 4, 3, 1) + 2 * hid
    # outside the fused kernel's nets: the three-kernel count
    for args in [(128, 4, 128, 128, "relu"), (128, 16, 128, 128, "relu"), (128, 4, 128, 16, "sine"),
                 (64, 5, 64, 16, "sigmoid"), (64, 0, 64, 16, "relu")]:
        assert not bench.fused_backward(*args)
        assert bench.train_bytes_per_row(*args) == bench.train_bytes_per_row(*args, fused=False)
    for args in [(64, 4, 3, 1, "sine"), (64, 4, 64, 16, "sigmoid"), (64, 4, 6, 16, "relu"),
                 (16, 1, 16, 16, "linear")]:
        assert bench.fused_backward(*args)


def test_one_kernel_training_bytes_per_row():
    """Widths 16, 32 and 64 with 2 to 5 matrices run the whole step in one
    kernel: X read (2 in) and T read (4 out) per row, nothing else."""
    for w, d in [(16, 1), (16, 4), (32, 2), (32, 4), (64, 1), (64, 4)]:
        assert bench.fused_step(w, d)
        assert bench.train_bytes_per_row(w, d, w, 16, "relu") == 2 * w + 64
        assert bench.train_bytes_per_row(w, d, 7, 3, "sine") == 14 + 12
    for w, d in [(16, 0), (16, 5), (32, 16), (64, 0), (64, 5), (128, 4)]:
        assert not bench.fused_step(w, d)


def test_default_steps_paper_protocol():
    """The bench's default step count follows section IV-A's rule,
    max(1000 * 2^18 / M, 250): 250 at 2^20 rows and above, 1000 at 2^18,
    4000 at 2^16."""
    import bench
    assert bench.default_steps(1 << 20) == 250
    assert bench.default_steps(1 << 22) == 250
    assert bench.default_steps(1 << 18) == 1000
    assert bench.default_steps(1 << 16) == 4000
    assert bench.default_steps(4096) == 64000
