"""C ABI checks that need no GPU: the library loads, exports every function nova.h declares,
the binding covers them, and the host-side logic (layouts, CU masks, argument validation)
behaves as documented."""
import ctypes as C
import os
import re

import pytest

from paper_2509_21301_amd import nova, synth

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "nova.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nova_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound():
    names = declared_functions()
    assert len(names) >= 20
    lib = C.CDLL(nova.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(nova._SIG), set(names) ^ set(nova._SIG)


def test_layouts_are_aligned_and_sized():
    (eo, eb), (lo, lb), (ho, hb) = nova.vit_layouts(synth.VIT_1008)
    for offs, total in [(eo, eb), (lo, lb), (ho, hb)]:
        assert all(o % 256 == 0 for o in offs) and total % 256 == 0
        assert offs == sorted(offs)
    H, I = 1280, 5120
    assert lb >= 2 * (4 * H * H + 2 * H * I)             # one layer of bf16 weights
    assert lb < 2 * (4 * H * H + 2 * H * I) + 12 * 256 + 2 * (9 * H + I)
    (lo, lb), (ho, hb) = nova.llm_layouts(synth.LLM_28)
    assert lb // 2 >= 3584 * (4608 + 3584 + 3 * 18944)
    assert hb // 2 >= 152064 * 3584


def test_invalid_configs_are_rejected():
    bad = [
        synth.VitConfig(hidden=256, heads=3, mlp=1024, layers=1, patch=4, merge=1, out_hidden=256, image_h=32, image_w=32),
        synth.VitConfig(hidden=256, heads=4, mlp=1024, layers=1, patch=4, merge=2, out_hidden=256, image_h=36, image_w=32),
        synth.VitConfig(hidden=96, heads=1, mlp=1024, layers=1, patch=4, merge=1, out_hidden=256, image_h=32, image_w=32),
    ]
    for cfg in bad:
        with pytest.raises(nova.NovaError):
            nova.vit_layouts(cfg)
    with pytest.raises(nova.NovaError):
        nova.llm_layouts(synth.LlmConfig(hidden=256, n_q=4, n_kv=3, head_dim=64, inter=688, vocab=4096, layers=1))
    with pytest.raises(nova.NovaError):
        nova.llm_layouts(synth.LlmConfig(hidden=256, n_q=4, n_kv=2, head_dim=64, inter=688, vocab=4096, layers=1, block=32))
    with pytest.raises(nova.NovaError) as e:
        nova.llm_layouts(synth.LlmConfig(hidden=256, n_q=4, n_kv=2, head_dim=96, inter=688, vocab=4096, layers=1))
    assert "head_dim" in str(e.value)


def test_cu_masks_follow_the_gfx950_bit_map():
    # bit i = 32 * slot + 8 * engine + xcd; n CUs = n/8 slots on every XCD, engines interleaved
    m = nova.make_cu_mask(32, 0)
    assert m == [0xFFFFFFFF] + [0] * 7
    m = nova.make_cu_mask(64, 8)
    assert m == [0, 0, 0xFFFFFFFF, 0xFFFFFFFF, 0, 0, 0, 0]
    m = nova.make_cu_mask(8, 0)                  # one CU per XCD, all on engine 0
    assert m == [0x000000FF] + [0] * 7
    m = nova.make_cu_mask(16, 1)                 # slots 1, 2: engines 1 and 2 of CU slot 0
    assert m == [0x00FFFF00] + [0] * 7
    full = nova.make_cu_mask(256, 0)
    assert full == [0xFFFFFFFF] * 8
    for n in range(32, 256, 32):
        a, b = nova.make_cu_mask(n, 0), nova.make_cu_mask(256 - n, n // 8)
        assert all((x & y) == 0 and (x | y) == 0xFFFFFFFF for x, y in zip(a, b))
    for bad in [(0, 0), (12, 0), (264, 0), (64, 28)]:
        with pytest.raises(nova.NovaError):
            nova.make_cu_mask(*bad)


def test_model_handles_and_workspace_sizes_on_host():
    # handles only validate and record pointers; fake 256-aligned addresses are never dereferenced
    fake = 1 << 20
    d = nova.VitDescC(nova.vit_config_c(synth.VIT_1008), fake, fake, fake, None, None, 0)
    h = C.c_void_p()
    nova._check(nova.lib.nova_vit_create(C.byref(d), C.byref(h)))
    ws1 = nova.lib.nova_vit_workspace_bytes(h, 1)
    ws8 = nova.lib.nova_vit_workspace_bytes(h, 8)
    assert ws1 > 5184 * 1280 * 4 and 7.5 * ws1 < ws8 < 8.5 * ws1
    nova.lib.nova_vit_destroy(h)
    d.embed = fake + 8                            # misaligned pointers are refused
    assert nova.lib.nova_vit_create(C.byref(d), C.byref(h)) == nova.EINVAL
    assert b"aligned" in nova.lib.nova_last_error()
    ld = nova.LlmDescC(nova.llm_config_c(synth.LLM_28), fake, fake, fake)
    nova._check(nova.lib.nova_llm_create(C.byref(ld), C.byref(h)))
    assert nova.lib.nova_kv_bytes(h, 100) == 28 * 100 * 4 * 16 * 128 * 2
    small = nova.lib.nova_llm_decode_workspace_bytes(h, 1, 2048)
    big = nova.lib.nova_llm_decode_workspace_bytes(h, 32, 2048)
    assert 0 < small < big
    assert nova.lib.nova_llm_prefill_workspace_bytes(h, 1500) > 1500 * 3584 * 4
    # argument checks happen before any device work
    kv = nova.KvC(fake, fake, 100)
    ws = fake
    rc = nova.lib.nova_llm_decode(h, fake, fake, fake, 8, 33, 100, C.byref(kv), fake, None, ws, big, None)
    assert rc == nova.EINVAL                      # batch 33 > 32
    rc = nova.lib.nova_llm_decode(h, fake, fake, fake, 4, 1, 100, C.byref(kv), fake, None, ws, big, None)
    assert rc == nova.ENOKV                       # 100 positions need 7 blocks > 4
    rc = nova.lib.nova_llm_decode(h, fake, fake, fake, 8, 1, 100, C.byref(kv), fake, None, ws, 16, None)
    assert rc == nova.ENOSPACE
    nova.lib.nova_llm_destroy(h)
