"""C ABI checks that need no GPU: the library loads, exports every function
that include/chimera.h declares, and its host-side sizing and validation
behave (no compute calls)."""
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "chimera.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(chimera_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    from paper_2402_15758_amd import binding
    L = binding.lib()
    names = declared_functions()
    assert len(names) >= 19
    for n in names:
        assert hasattr(L, n), n


def _cfg(mc, max_positions=4096):
    from paper_2402_15758_amd import binding as B
    return B.chimera_config(mc.n_layers, mc.d_model, mc.n_heads, mc.head_dim, mc.d_ffn, mc.vocab,
                            mc.n_draft_heads, mc.rope_base, mc.rms_eps,
                            B.CHIMERA_BF16 if mc.dtype == "bf16" else B.CHIMERA_F32, max_positions)


@pytest.mark.parametrize("mc", [synth.TINY, synth.LLAMA7B, synth.LLAMA13B])
def test_weight_bytes_cover_every_tensor(mc):
    from paper_2402_15758_amd import binding as B
    got = B.chimera_weight_bytes(_cfg(mc))
    es = 2 if mc.dtype == "bf16" else 4
    want = 0
    for name, shape, group in synth.tensor_specs(mc):
        n = 1
        for s in shape:
            n *= s
        want += n * (4 if group == "gain" else es)
    want += 2 * 4096 * (mc.head_dim // 2) * 4  # rotary tables
    assert want <= got <= want + 256 * (len(synth.tensor_specs(mc)) + 8)


def test_config_validation_errors():
    from paper_2402_15758_amd import binding as B
    bad = _cfg(synth.TINY)
    bad.head_dim = 96
    with pytest.raises(B.ChimeraError) as e:
        B.chimera_weight_bytes(bad)
    assert e.value.status == -1 and "head_dim" in str(e.value)
    bad = _cfg(synth.TINY)
    bad.n_heads = 3
    with pytest.raises(B.ChimeraError):
        B.chimera_weight_bytes(bad)


def test_tree_arrays():
    from paper_2402_15758_amd.runtime import tree_arrays
    parent, rank = tree_arrays(synth.TREE_T8)
    assert list(parent) == [-1, 0, 0, 0, 1, 1, 2, 4]
    assert list(rank) == [0, 0, 1, 2, 0, 3, 0, 0]


def test_load_refuses_host_tensors_before_any_device_work():
    """chimera_load reads device memory only: a host tensor is refused while
    the tensor list is validated, before anything is copied or launched."""
    import numpy as np
    from paper_2402_15758_amd import binding as B
    mc = synth.TINY
    emb = np.zeros(mc.vocab * mc.d_model, dtype=np.float32)
    t = (B.chimera_tensor * 1)(B.chimera_tensor(b"tok_embed", emb.ctypes.data, emb.size, B.CHIMERA_F32, 0))
    with pytest.raises(B.ChimeraError) as e:
        B.chimera_load(_cfg(mc), list(t), 256, 1 << 40, 0)
    assert e.value.status == B.CHIMERA_EINVAL and "not in device memory" in str(e.value)
