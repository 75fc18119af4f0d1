"""The forward GEMM's chunk pipeline, walked on the CPU for every chunk count
the d_in splits can give (1 .. 48): two register sets and two LDS buffers,
chunks loaded kDepth ahead with indices clamped to the last chunk, a
branch-free steady loop and a guarded tail, as in k_mlp_fwd_sk
(paper_2211_00889_amd/csrc/mlp.hip).  Checks that every chunk is multiplied
exactly once, in order, from the buffer it was staged into, that a register
set is only refilled after it was staged, and that a buffer is only
restaged after the barrier that follows its last multiply."""
import pytest

K_DEPTH = 2


def walk(nck, depth=K_DEPTH, mistake=False):
    regs = [None] * depth          # chunk held by each register set
    staged_from = {}               # chunk -> register-set contents when staged
    buf = [None, None]             # chunk held by each LDS buffer
    reads_since_barrier = set()    # buffers multiplied since the last barrier
    multiplied = []
    events = []

    def load(r, c):
        assert regs[r] is None or regs[r] == "staged", f"set {r} refilled before staging"
        regs[r] = c

    def stage(r, b):
        c = regs[r]
        assert c is not None and c != "staged"
        assert b not in reads_since_barrier, f"buffer {b} restaged before the barrier"
        buf[b] = c
        staged_from[c] = b
        regs[r] = "staged"

    def multiply(b, c):
        assert buf[b] == min(c, nck - 1) == c, f"chunk {c} multiplied from buffer {b} holding {buf[b]}"
        reads_since_barrier.add(b)
        multiplied.append(c)

    def barrier():
        reads_since_barrier.clear()

    # prologue
    for c in range(depth):
        load(c, min(c, nck - 1))
    stage(0, 0)
    load(0, min(depth, nck - 1))
    barrier()

    def step(c, r):
        multiply(c & 1, c)
        if c + 1 < nck:
            stage(r, (c + 1) & 1)
        if c + 1 + depth < nck:
            load(r, c + 1 + depth)
        barrier()

    c = 0
    while c + 2 * depth < nck:          # steady state, every step stages and loads
        for j in range(depth):
            multiply((c + j) & 1, c + j)
            stage((j + 1) % depth, (c + j + (0 if mistake else 1)) & 1)
            load((j + 1) % depth, c + j + 1 + depth)
            barrier()
        c += depth
    while c < nck:
        for j in range(depth):
            if c + j < nck:
                step(c + j, (j + 1) % depth)
        c += depth
    return multiplied, staged_from


@pytest.mark.parametrize("nck", range(1, 49))
def test_every_chunk_multiplied_once_in_order(nck):
    multiplied, staged_from = walk(nck)
    assert multiplied == list(range(nck))
    assert all(staged_from[c] == (c & 1) for c in range(nck))


def test_a_planted_mistake_is_caught():
    """Staging the next chunk into the buffer being multiplied (a planted
    mistake in the steady loop) fails the walk wherever that loop runs."""
    for nck in range(1, 49):
        if nck <= 2 * K_DEPTH:
            walk(nck, mistake=True)      # the steady loop does not run
            continue
        with pytest.raises(AssertionError):
            walk(nck, mistake=True)
