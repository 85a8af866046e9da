"""The microbenchmark kernels: the copy moves the bytes, the hand-over and
barrier loops complete and report positive times."""
import pytest

pytestmark = pytest.mark.gpu


def test_copy_moves_every_byte(gpu):
    import torch

    from paper_1508_00703_amd import native

    for nbytes in (16, 4096 + 16, 3 * 1024 * 1024):
        src = torch.randint(0, 2 ** 31 - 1, (nbytes // 4,), dtype=torch.int32, device=gpu)
        dst = torch.zeros_like(src)
        native.pdb_mb_copy(src, dst)
        torch.cuda.synchronize()
        assert torch.equal(src, dst)
    odd = torch.zeros(3, dtype=torch.int32, device=gpu)
    with pytest.raises(native.PdbError):
        native.pdb_mb_copy(odd, odd)


@pytest.mark.parametrize("partner", [1, 8, 255])
def test_hop_round_trips(gpu, partner):
    from paper_1508_00703_amd import native

    ns, xa, xb = native.pdb_mb_hop(2000, partner, gpu)
    assert 10.0 < ns < 1e6
    assert 0 <= xa < 16 and 0 <= xb < 16


@pytest.mark.parametrize("blocks", [2, 64])
def test_barrier_rounds(gpu, blocks):
    from paper_1508_00703_amd import native

    ns = native.pdb_mb_barrier(500, blocks, gpu)
    assert 10.0 < ns < 1e7
