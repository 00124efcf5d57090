"""CPU checks of the C ABI: the library loads, exports every entry point the
header declares, and the host-only size query and config validation behave
as documented.  No call here touches a GPU."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2604_20919_amd import sdverify as sv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sd_verify.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:sd_status|const char\*)\s+(sd_\w+)\(", src, re.M)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("sd_verify_init", "sd_verify_batch", "sd_accept"):
        assert n in names
    assert set(names) == set(sv.EXPORTS)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", sv.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (sd_\w+)$", out, re.M))
    missing = set(_declared()) - exported
    assert not missing, missing
    lib = sv.lib()
    for n in _declared():
        assert hasattr(lib, n)


def test_status_strings():
    assert sv.status_str(sv.SD_OK) == "ok"
    assert "pages" in sv.status_str(sv.SD_ENOMEM)
    assert sv.status_str(12345) == "unknown status"


def _cfg(**kw):
    base = dict(n_layers=64, d_model=5120, n_q_heads=64, n_kv_heads=8, head_dim=128, d_ffn=25600,
                vocab=151936, qk_norm=1, dtype=sv.SD_BF16, n_pages=4096, max_users=16, max_draft=4,
                max_batch_users=16, max_batch_tokens=80, max_ctx=1029, max_pending=2)
    base.update(kw)
    return sv.make_config(**base)


def test_query_sizes_32b_shape():
    kv, ws, wp = sv.sd_verify_query_sizes(_cfg())
    # projection matrices + lm_head of the 32B shape in bf16
    per_layer = 10240 * 5120 + 5120 * 8192 + 2 * 25600 * 5120 + 5120 * 25600
    assert wp == (64 * per_layer + 151936 * 5120) * 2
    # 64 layers x 4096 pages x (K + V) x 8 heads x 16 tokens x 128 x 2 bytes
    assert kv == 64 * 4096 * 2 * 8 * 16 * 128 * 2
    assert ws % 256 == 0 and ws > 0
    # logits of 80 slots x 151936 fp32 alone need 48.6 MB per pending batch
    assert ws > 2 * 80 * 151936 * 4


@pytest.mark.parametrize("bad", [
    dict(n_q_heads=60), dict(page_tokens=8), dict(max_pending=9), dict(max_draft=0),
    dict(dtype=7), dict(qk_norm=2), dict(n_pages=0), dict(max_batch_tokens=1),
])
def test_query_sizes_rejects_bad_configs(bad):
    cfg = _cfg(**{k: v for k, v in bad.items() if k != "page_tokens"})
    if "page_tokens" in bad:
        cfg.page_tokens = bad["page_tokens"]
    with pytest.raises(sv.SdError) as e:
        sv.sd_verify_query_sizes(cfg)
    assert e.value.status == sv.SD_EINVAL


def test_query_sizes_unsupported_bf16_shapes():
    with pytest.raises(sv.SdError) as e:
        sv.sd_verify_query_sizes(_cfg(head_dim=64))
    assert e.value.status == sv.SD_ENOTIMPL
    with pytest.raises(sv.SdError) as e:
        sv.sd_verify_query_sizes(_cfg(max_batch_tokens=512))
    assert e.value.status == sv.SD_ENOTIMPL


def test_null_arguments_are_rejected_without_a_device():
    lib = sv.lib()
    assert lib.sd_verify_query_sizes(None, None, None, None) == sv.SD_EINVAL
    out = ctypes.c_void_p()
    assert lib.sd_verify_init(None, None, None, None, None, ctypes.byref(out)) == sv.SD_EINVAL
    assert lib.sd_accept(None, 0, None, None, 0) == sv.SD_EINVAL
    assert lib.sd_verify_batch(None, 0, 1, None, None, None, None, 0, 0, 0, None, None) == sv.SD_EINVAL
    assert lib.sd_verify_destroy(None) == sv.SD_EINVAL


def test_noalloc_limits_are_checked_before_any_device_call():
    """sd_sample_logits_noalloc refuses arguments on the host, before it
    looks up its scratch array or enqueues anything."""
    lib = sv.lib()
    u = (ctypes.c_int32 * 65)(*range(65))
    L = (ctypes.c_int32 * 65)(*([1] * 65))
    p = ctypes.c_void_p(16)  # never dereferenced: every call below is refused first
    assert lib.sd_sample_logits_noalloc(65, u, L, 16, p, p, p, 0, 0, 0, None, p, None) == sv.SD_ELIMIT
    L2 = (ctypes.c_int32 * 2)(512, 511)  # 1025 slots
    assert lib.sd_sample_logits_noalloc(2, u, L2, 16, p, p, p, 0, 0, 0, None, p, None) == sv.SD_ELIMIT
    assert lib.sd_sample_logits_noalloc(1, u, L, sv.SD_NOALLOC_MAX_VOCAB + 1, p, p, p, 0, 0, 0, None, p,
                                        None) == sv.SD_ELIMIT
    assert lib.sd_sample_logits_noalloc(0, u, L, 16, p, p, p, 0, 0, 0, None, p, None) == sv.SD_EINVAL
    assert lib.sd_sample_logits_noalloc(1, u, L, 16, p, None, p, 1, 0, 0, None, p, None) == sv.SD_EINVAL
    assert lib.sd_sample_logits_noalloc(1, u, L, 16, p, p, p, 3, 0, 0, None, p, None) == sv.SD_EINVAL
    assert sv.status_str(sv.SD_ELIMIT) != "unknown status"


def test_query_sizes_rejects_a_layer_of_pages_beyond_4gb():
    """The attention kernel addresses one layer's pages with 32-bit offsets:
    65535 pages of the 32B shape (64 KB each) pass, 65536 do not."""
    sv.sd_verify_query_sizes(_cfg(n_pages=65535))
    with pytest.raises(sv.SdError) as e:
        sv.sd_verify_query_sizes(_cfg(n_pages=65536))
    assert e.value.status == sv.SD_ENOTIMPL
