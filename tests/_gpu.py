"""Shared GPU-test plumbing.  Importing the binding raises if the HIP library
is not built, so a GPU run never passes on a missing extension."""
import torch

from paper_2608_01150_amd import api  # noqa: F401  (raises ImportError if libzl_attn.so is missing)

HAVE_GPU = torch.cuda.is_available()


def to64(t):
    return t.detach().float().cpu().double().numpy()
