"""The binding rejects arguments the kernel would misuse before anything is
launched (outputs the kernel writes B entries of, devices, dtypes), and
accepts a workspace of any element type whose byte size suffices."""
import pytest
import torch

from paper_2406_11016_amd import binding
from paper_2406_11016_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def inputs():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    binding.load_library()
    x = W.small_case(4, 3, 1000, "f32", seed=3)
    return x, binding.to_device(x, "cuda")


def test_output_shapes_and_dtypes_are_checked(inputs):
    x, (d, t, tok, u) = inputs
    bad = [dict(accepted_len=torch.empty(3, dtype=torch.int32, device="cuda")),
           dict(next_token=torch.empty(4, dtype=torch.int64, device="cuda")),
           dict(accepted_len=torch.empty(4, dtype=torch.int32)),
           dict(next_token=torch.empty(8, dtype=torch.int32, device="cuda")[::2])]
    for kw in bad:
        with pytest.raises(binding.SpecVerifyError):
            binding.verify(d, t, tok, u, **kw)
    with pytest.raises(binding.SpecVerifyError):
        binding.verify(d, t, tok.cpu(), u)
    with pytest.raises(binding.SpecVerifyError):
        binding.verify(d, t, tok, u, gammas=torch.full((4,), 2, dtype=torch.int64, device="cuda"))


def test_workspace_of_any_element_type(inputs):
    x, (d, t, tok, u) = inputs
    need = binding.workspace_bytes(x.batch, x.gamma, x.vocab, d.dtype)
    ws32 = torch.zeros((need + 3) // 4, dtype=torch.float32, device="cuda")
    a0, n0 = binding.verify(d, t, tok, u)
    a1, n1 = binding.verify(d, t, tok, u, workspace=ws32)
    torch.cuda.synchronize()
    assert torch.equal(a0, a1) and torch.equal(n0, n1)
    with pytest.raises(binding.SpecVerifyError):
        binding.verify(d, t, tok, u, workspace=torch.zeros(need // 8, dtype=torch.float32, device="cuda"))
