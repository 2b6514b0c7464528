"""The C ABI library loads, exports what include/m2r2.h declares, and rejects
bad arguments before touching a device (no GPU needed)."""
import ctypes
import os
import re
import subprocess

import pytest

import synth
from paper_2502_02040_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header=None):
    """Entry points declared in include/<header> (every header if None)."""
    names = set()
    for h in ([header] if header else sorted(os.listdir(os.path.join(ROOT, "include")))):
        if h.endswith(".h"):
            src = open(os.path.join(ROOT, "include", h)).read()
            names |= set(re.findall(r"M2R2_API\s+[\w\s\*]+?\b(m2r2_\w+)\s*\(", src))
    return names


# the calls the decode path's boundary is built around: create/destroy and
# the workspace size, one decode step, the draft, the verification, the
# expert prefetch, and the error reporting
CORE = {"m2r2_workspace_size", "m2r2_create", "m2r2_destroy", "m2r2_decode_step", "m2r2_draft", "m2r2_verify",
        "m2r2_prefetch_experts", "m2r2_last_error", "m2r2_sync_check"}
# declared extensions of the boundary (each with its reason in the header)
EXTENSIONS = {"m2r2_device_errors", "m2r2_expert_bytes", "m2r2_pack_expert", "m2r2_moe_set_policy",
              "m2r2_moe_reset", "m2r2_moe_stats", "m2r2_expert_cache_replay", "m2r2_moe_set_preload_table",
              "m2r2_set_arla",
              # the decode step for callers that cannot allocate (scratch in a static device array)
              "m2r2_decode_step_noalloc"}


def test_header_declarations_match_binding():
    assert _declared("m2r2.h") == set(binding.EXPORTS) == CORE | EXTENSIONS
    assert _declared("m2r2_measure.h") == set(binding.MEASURE_EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = binding.lib()
    for name in _declared():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (m2r2_\w+)", out))
    assert exported == _declared()


def test_workspace_size_and_validation():
    cfg = synth.CONFIGS["phi3"]
    n = binding.workspace_size(cfg, 1, 16, 1536)
    # the workspace holds the tile-packed projection matrices (bf16) plus scratch
    d, q, F, V, L = cfg.d_model, cfg.qdim, cfg.ffn, cfg.vocab, cfg.n_layers
    packed = 2 * (L * (3 * q * d + 16 * d + d * q + 3 * F * d) + V * d)
    assert packed < n < packed + (64 << 20)
    assert binding.workspace_size(cfg, 8, 16, 4352) >= n
    with pytest.raises(binding.M2R2Error) as e:
        binding.workspace_size(cfg.replace(head_dim=80), 1, 16, 1024)
    assert e.value.status == -7
    with pytest.raises(binding.M2R2Error) as e:
        binding.workspace_size(cfg, 9, 16, 1024)
    assert e.value.status == -2
    with pytest.raises(binding.M2R2Error) as e:
        binding.workspace_size(cfg.replace(d_model=3000), 1, 16, 1024)
    assert e.value.status == -2


def test_null_arguments_are_rejected():
    lib = binding.lib()
    assert lib.m2r2_decode_step(None, 1, 1, None, None, None, None, None, None) == -1
    assert b"ctx" in lib.m2r2_last_error()
    assert lib.m2r2_verify(None, None, 1, None, None, None, None, None, None) == -1
    assert lib.m2r2_draft(None, None, None, 1, 1, None, None, None) == -1
    cfg = binding.make_config(synth.CONFIGS["tiny"])
    out = ctypes.c_void_p()
    assert lib.m2r2_create(ctypes.byref(cfg), None, 1, 16, 128, None, 0, ctypes.byref(out)) == -1
    assert lib.m2r2_set_arla(None, None) == -1
    assert lib.m2r2_moe_set_policy(None, 0) == -1
    assert lib.m2r2_moe_set_preload_table(None, None, 1) == -1
    assert lib.m2r2_sync_check(None, None) == -1
    assert lib.m2r2_decode_step_noalloc(None, 1, 1, None, None, None, None, None, None) == -1
