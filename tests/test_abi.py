"""The C ABI library loads, exports every function include/seed.h declares, and rejects bad
configurations on the host (no GPU work is done in these tests)."""
import ctypes
import os
import re

import pytest

from paper_2609_36590_amd import binding, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    text = open(os.path.join(ROOT, "include", "seed.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(seed_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.lib_path()):
        pytest.fail("library not built: run __graft_entry__.build() first")
    return binding.load_library()


def test_exports_every_declared_function(lib):
    declared = _header_functions()
    assert "seed_generate" in declared and len(declared) >= 12
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(binding.EXPORTS) == declared


def test_struct_sizes_match_header_layout():
    assert ctypes.sizeof(binding.SeedConfig) == 15 * 4
    assert ctypes.sizeof(binding.SeedTensor) == 8 + 8 + 4 * 3 + 4 + 16
    assert ctypes.sizeof(binding.SeedGenOpts) == 16 + 8 + 8
    assert ctypes.sizeof(binding.SeedStats) == 3 * 8 + 2 * 8 + 8 + 8 + 2 * 8


def _cfg(**kw):
    c = binding.make_config(synth.C1_TINY, 1, 128, 4)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_arena_bytes_scale_with_capacity(lib):
    w1, kv1, ws1 = binding.seed_arena_bytes(_cfg())
    w2, kv2, ws2 = binding.seed_arena_bytes(_cfg(max_ctx=256))
    assert w2 > w1 and kv2 > kv1 and ws2 > ws1
    # the 4B-scale weights take 8.05 GB in bf16 (tied head counted once)
    big = binding.make_config(synth.C3_4B, 1, 1545, 4)
    w, kv, ws = binding.seed_arena_bytes(big)
    assert 8.0e9 < w < 8.1e9
    # KV: 36 layers x 2 x 8 heads x 128 dims x 2 bytes per position, in 16-position blocks
    assert kv >= 36 * 2 * 8 * 128 * 2 * 1545


@pytest.mark.parametrize("field,value,status", [
    ("hidden", 250, -5), ("head_dim", 96, -5), ("kv_block", 32, -5), ("n_dec_layers", 9, -1),
    ("dtype", 7, -1), ("max_batch", 0, -5), ("max_draft", 16, -5), ("vocab", 1000, -5),
    ("n_kv_heads", 3, -5), ("max_ctx", 1, -1),
])
def test_invalid_configs_are_rejected(lib, field, value, status):
    with pytest.raises(binding.SeedError) as e:
        binding.seed_arena_bytes(_cfg(**{field: value}))
    assert e.value.status == status
    assert lib.seed_last_error().decode()


def test_batch_times_rows_limit(lib):
    with pytest.raises(binding.SeedError) as e:
        binding.seed_arena_bytes(_cfg(max_batch=8, max_draft=8))
    assert "64" in str(e.value)


def test_null_arguments(lib):
    assert lib.seed_arena_bytes(None, None, None, None) == -1
    assert lib.seed_create(None, None, None, None, None, None) == -1
    assert lib.seed_prefill(None, 1, None, None) == -1
    assert lib.seed_draft(None, 1, None, None) == -1
    assert lib.seed_verify(None, 1, None, None, None, None) == -1
    assert lib.seed_generate(None, 1, None, None, None, None, None, None) == -1
    assert lib.seed_read_kv(None, 0, 0, 0, 1, None, None) == -1
    lib.seed_destroy(None)


def test_spec_cache_bytes_cover_the_decoder_layers(lib):
    c = binding.make_config(synth.C3_4B, 1, 1545, 4)
    n = binding.seed_spec_kv_bytes(c)
    # 2 decoder layers x 2 (K, V) x 8 heads x 128 dims x 2 bytes per position
    assert n >= 2 * 2 * 8 * 128 * 2 * 1545
    assert n < 1.1 * 2 * 2 * 8 * 128 * 2 * (1545 + 16)


def test_tree_options_layout_and_paper_defaults(lib):
    # float tau, int max_depth, int n_levels, float thr[4], int k[4], int k_rest, int max_nodes
    assert ctypes.sizeof(binding.SeedTreeOpts) == 4 * (3 + 4 + 4 + 2)
    o = binding.tree_opts(6)
    assert o.tau == pytest.approx(0.7) and o.max_depth == 6 and o.n_levels == 3
    assert [o.thr[j] for j in range(3)] == pytest.approx([0.95, 0.8, 0.5])
    assert list(o.k[:3]) == [1, 3, 5] and o.k_rest == 10 and o.max_nodes == 64
    o2 = binding.tree_opts(3, tau=0.5, table=((0.9, 2),), rest=4, max_nodes=20)
    assert (o2.tau, o2.n_levels, o2.k[0], o2.k_rest, o2.max_nodes) == (pytest.approx(0.5), 1, 2, 4, 20)
    assert o2.thr[0] == pytest.approx(0.9)


def test_struct_offsets_match_the_c_compiler(tmp_path):
    """Every field offset of the ctypes structures equals the C compiler's for include/seed.h."""
    import subprocess
    structs = {"seed_config": binding.SeedConfig, "seed_gen_opts": binding.SeedGenOpts,
               "seed_stats": binding.SeedStats, "seed_tree_opts": binding.SeedTreeOpts}
    src = ['#include <stdio.h>', '#include <stddef.h>', '#include "seed.h"', "int main(void) {"]
    for c_name, cls in structs.items():
        src.append(f'  printf("{c_name} %zu\\n", sizeof({c_name}));')
        for f, _ in cls._fields_:
            src.append(f'  printf("{c_name}.{f} %zu\\n", offsetof({c_name}, {f}));')
    src.append("  return 0;\n}")
    (tmp_path / "layout.c").write_text("\n".join(src))
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(tmp_path / "layout.c"), "-o",
                    str(tmp_path / "layout")], check=True)
    got = dict(line.split() for line in subprocess.run([str(tmp_path / "layout")], check=True, capture_output=True,
                                                        text=True).stdout.splitlines())
    for c_name, cls in structs.items():
        assert int(got[c_name]) == ctypes.sizeof(cls), c_name
        for f, _ in cls._fields_:
            assert int(got[f"{c_name}.{f}"]) == getattr(cls, f).offset, (c_name, f)
