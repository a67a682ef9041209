"""The product path has no fallback (CPU): without the HIP library, with host
tensors, or without a GPU, the binding raises instead of computing anything
elsewhere; and no module of the package imports the oracle."""
import ast
import os

import pytest
import torch

from paper_2509_20883_amd import recis as R

PKG = os.path.dirname(os.path.abspath(R.__file__))


def test_missing_library_raises(monkeypatch):
    monkeypatch.setattr(R, "LIB_PATH", os.path.join(PKG, "no_such_library.so"))
    monkeypatch.setattr(R, "_lib", None)
    with pytest.raises(R.RecisError, match="not built"):
        R.lib()


def test_host_tensors_are_rejected():
    with pytest.raises(R.RecisError, match="on the GPU"):
        R.fused_mod(torch.zeros(4, dtype=torch.int64), torch.tensor([0, 4]), torch.tensor([3]))
    with pytest.raises(R.RecisError, match="on the GPU"):
        R.fused_bucketize(torch.zeros(4), torch.tensor([0, 4]), torch.tensor([0.5]), torch.tensor([0, 1]))


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the behaviour without a GPU")
def test_table_without_gpu_raises():
    with pytest.raises((R.RecisError, RuntimeError)):
        R.Table(16)


def test_package_does_not_import_the_oracle():
    for name in os.listdir(PKG):
        if not name.endswith(".py"):
            continue
        with open(os.path.join(PKG, name)) as fh:
            tree = ast.parse(fh.read(), filename=name)
        for node in ast.walk(tree):
            mods = []
            if isinstance(node, ast.Import):
                mods = [a.name for a in node.names]
            elif isinstance(node, ast.ImportFrom):
                mods = [node.module or ""]
            assert not any(m == "oracle" or m.startswith("oracle.") for m in mods), f"{name} imports the oracle"
