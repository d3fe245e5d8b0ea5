"""Host-side checks of the HIP library that need no GPU: it loads, exports
every function include/mlip.h declares, counts weights like the blob layout,
and rejects invalid arguments before touching the device."""
import ctypes
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def binding():
    lib = os.path.join(ROOT, "paper_2608_16329_amd", "libmlip.so")
    if not os.path.exists(lib):
        from paper_2608_16329_amd import build
        build.build()
    from paper_2608_16329_amd import binding as b
    return b


def _declared():
    with open(os.path.join(ROOT, "include", "mlip.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mlip_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol(binding):
    declared = _declared()
    assert declared, "no declarations parsed"
    lib = ctypes.CDLL(binding.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(binding.EXPORTED) == declared


@pytest.mark.parametrize("over", [{}, {"n_species": 6}, {"n_species": 3, "enc_cond": 1}, {"reg_cond": 0},
                                  {"k": 16, "lmax": 1}, {"enc_hidden": 5, "reg_hidden": 2, "angular": 1}])
def test_weight_count_matches_blob_layout(binding, over):
    hp = synth.HParams(n_species=2)
    for k, v in over.items():
        setattr(hp, k, v)
    assert binding.mlip_weight_count(hp) == synth.weight_count(hp)


def test_invalid_hparams(binding):
    for over in ({"n_species": 0}, {"k": 0}, {"enc_cond": 3}, {"reg_hidden": 0}, {"angular": 2}):
        hp = synth.HParams(n_species=2)
        for k, v in over.items():
            setattr(hp, k, v)
        assert binding.mlip_weight_count(hp) == 0


@pytest.mark.parametrize("over", [{"k": 24}, {"lmax": 6}, {"angular": 1, "lmax": 4}, {"angular": 1, "k": 16},
                                  {"angular": 1, "k": 64}, {"enc_width": 64},
                                  {"reg_width": 32}, {"precision": 16}, {"n_species": 17}, {"enc_hidden": 9}])
def test_create_rejects_unsupported_before_device(binding, over):
    hp = synth.HParams(n_species=2)
    for k, v in over.items():
        setattr(hp, k, v)
    w = synth.random_weights(hp, 0) if binding.mlip_weight_count(hp) else [0.0]
    with pytest.raises(binding.MlipError, match="ARG: (unsupported|invalid)"):
        binding.mlip_create(hp, w)


def test_create_rejects_wrong_weight_count(binding):
    hp = synth.HParams(n_species=2)
    with pytest.raises(binding.MlipError, match="ARG.*n_weights"):
        binding.mlip_create(hp, synth.random_weights(hp, 0)[:-1])


def test_null_context_is_safe(binding):
    lib = binding._lib
    assert isinstance(lib.mlip_last_error(None), bytes)
    lib.mlip_destroy(None)
    assert lib.mlip_compute(None, None, None, None, None, None) == -1
    assert lib.mlip_build_neighbors(None, 1, None, None, None) == -1
