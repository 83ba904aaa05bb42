"""Plant plausible mistakes in a COPY of the CPU oracle and check that the pins
in test_oracle_pins.py catch every one of them.

Each mutant is a textual edit of kvoracle.c compiled into a temporary library;
the pin suite then runs in a subprocess against it (KVO_ORACLE_LIB) and must
fail.  The committed oracle is never modified.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "kvoracle.c")

# (name, original text, replacement, occurrence to replace: None = all)
MUTANTS = [
    ("drop_in_page_offset_load",
     "slot = pool_page * page_size + t % page_size;\n        memcpy(pool_slab",
     "slot = pool_page * page_size;\n        memcpy(pool_slab", None),
    ("page_not_scaled",
     "slots_out[t] = pool_page * page_size + in_page;",
     "slots_out[t] = pool_page + in_page;", None),
    ("swap_k_v_in_host_offset",
     "return (((int64_t)layer * 2 + kv) * host_tokens + token) * row_bytes;",
     "return (((int64_t)layer * 2 + (1 - kv)) * host_tokens + token) * row_bytes;", None),
    ("stride_num_tokens_not_host_tokens",
     "kvo_host_row_offset(l, kv, host_tokens[s], 0, row_bytes);",
     "kvo_host_row_offset(l, kv, num_tokens[s], 0, row_bytes);", None),
    ("div_mod_swapped",
     "int64_t pool_page = page_idx[t / page_size];\n        int64_t slot;\n        if (pool_page < 0 || pool_page >= num_pages)\n            return KVO_ERANGE;\n        slot = pool_page * page_size + t % page_size;\n        memcpy(pool_slab",
     "int64_t pool_page = page_idx[t % page_size];\n        int64_t slot;\n        if (pool_page < 0 || pool_page >= num_pages)\n            return KVO_ERANGE;\n        slot = pool_page * page_size + t / page_size;\n        memcpy(pool_slab", None),
    ("drop_last_row_load",
     "for (t = 0; t < num_tokens; ++t) {\n        int64_t pool_page = page_idx[t / page_size];\n        int64_t slot;\n        if (pool_page < 0 || pool_page >= num_pages)\n            return KVO_ERANGE;\n        slot = pool_page * page_size + t % page_size;\n        memcpy(pool_slab",
     "for (t = 0; t + 1 < num_tokens; ++t) {\n        int64_t pool_page = page_idx[t / page_size];\n        int64_t slot;\n        if (pool_page < 0 || pool_page >= num_pages)\n            return KVO_ERANGE;\n        slot = pool_page * page_size + t % page_size;\n        memcpy(pool_slab", None),
    ("v_never_moved",
     "for (kv = 0; kv < 2; ++kv) {\n                uint8_t *slab",
     "for (kv = 0; kv < 1; ++kv) {\n                uint8_t *slab", None),
    ("offload_row_stride_wrong",
     "memcpy(host_slab + t * row_bytes, pool_slab + slot * row_bytes, (size_t)row_bytes);",
     "memcpy(host_slab + t * row_bytes, pool_slab + t * row_bytes, (size_t)row_bytes);", None),
    ("no_duplicate_check",
     "if (written[slot / 8] & (uint8_t)(1u << (slot % 8))) {",
     "if (0) {", None),
    ("page_first_layer_page_swapped",
     "return (((page * num_layers + layer) * 2 + kv) * page_size + in_page) * row_bytes;",
     "return (((layer * num_layers + page) * 2 + kv) * page_size + in_page) * row_bytes;", None),
    ("page_first_in_page_dropped",
     "return (((page * num_layers + layer) * 2 + kv) * page_size + in_page) * row_bytes;",
     "return (((page * num_layers + layer) * 2 + kv) * page_size) * row_bytes;", None),
    ("head_major_head_token_swapped",
     "return ((((int64_t)layer * 2 + kv) * num_heads + head) * host_tokens + token) * seg_bytes;",
     "return ((((int64_t)layer * 2 + kv) * host_tokens + token) * num_heads + head) * seg_bytes;", None),
    ("head_major_pool_segment_offset_dropped",
     "memcpy(prow + h * seg, hseg, (size_t)seg);",
     "memcpy(prow, hseg, (size_t)seg);", None),
    ("layer_end_inclusive_check",
     "layer_end > num_layers || layer_begin >= layer_end)\n        return KVO_EINVAL;\n    if (n_spans > 0 && (host == NULL || host_tokens == NULL || num_tokens == NULL || page_idx == NULL))\n        return KVO_EINVAL;\n    rc = kvo_check_batch(n_spans, host_tokens, num_tokens, page_idx, num_slots, page_size, 1);",
     "layer_end > num_layers + 1 || layer_begin > layer_end)\n        return KVO_EINVAL;\n    if (n_spans > 0 && (host == NULL || host_tokens == NULL || num_tokens == NULL || page_idx == NULL))\n        return KVO_EINVAL;\n    rc = kvo_check_batch(n_spans, host_tokens, num_tokens, page_idx, num_slots, page_size, 1);", None),
]


@pytest.mark.parametrize("name,old,new,occ", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new, occ):
    src = open(SRC).read()
    assert old in src, f"mutant {name}: anchor text not found in the oracle"
    mutated = src.replace(old, new)
    assert mutated != src
    c = tmp_path / "mutant.c"
    c.write_text(mutated)
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-std=c99", "-O1", "-fPIC", "-shared", str(c), "-o", str(lib)], check=True)
    env = dict(os.environ, KVO_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_layouts.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"


# Mutants of the copy's arithmetic (not of its input validation, which the
# property tests never exercise): the hypothesis-drawn properties alone must
# catch each of them too.
VALIDATION_MUTANTS = {"no_duplicate_check", "layer_end_inclusive_check"}


@pytest.mark.parametrize("name,old,new,occ", [m for m in MUTANTS if m[0] not in VALIDATION_MUTANTS],
                         ids=[m[0] for m in MUTANTS if m[0] not in VALIDATION_MUTANTS])
def test_properties_catch_arithmetic_mutant(tmp_path, name, old, new, occ):
    mutated = open(SRC).read().replace(old, new)
    c = tmp_path / "mutant.c"
    c.write_text(mutated)
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-std=c99", "-O1", "-fPIC", "-shared", str(c), "-o", str(lib)], check=True)
    env = dict(os.environ, KVO_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_properties.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} survived the property tests:\n{r.stdout[-2000:]}"
