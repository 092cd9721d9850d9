"""The C-ABI library without a GPU: it loads, exports every entry point that
include/marche.h declares, and rejects bad arguments on the host before any
HIP call (CPU only; no kernel is launched)."""
import ctypes as C
import os
import re

import pytest

from paper_2506_12035_amd import binding, build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "marche.h")
FAKE = 0x10000000  # never dereferenced: validation fails first


@pytest.fixture(scope="module", autouse=True)
def built_library():
    if not os.path.exists(binding.LIB_PATH):
        build.build()
    return binding.lib()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return set(re.findall(r"^\s*(?:const\s+)?(?:marche_status_t|size_t|int32_t|void|char)\s*\**\s*(\w+)\s*\(",
                          text, flags=re.M))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert {"kv_cache_init", "marche_step", "select_refresh"} <= names
    assert names == set(binding.EXPORTED)
    lib = C.CDLL(binding.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def _model(**kw):
    base = dict(n_layers=2, d_model=1024, n_heads=16, head_dim=64, d_mlp=4096, n_tokens=320,
                dtype=binding.MARCHE_BF16, ln_eps=1e-6)
    base.update(kw)
    return binding.make_model(**base)


def _cache(m, batch=2):
    return binding.KVCache(FAKE, FAKE, m.n_layers, batch, m.n_heads, m.n_tokens, m.head_dim, m.dtype)


def _layers(n):
    return binding.make_layers([{k: FAKE for k, _ in binding.Layer._fields_} for _ in range(n)])


def _step(m, cache=None, layers=None, **kw):
    args = dict(layer_begin=0, layer_end=m.n_layers, batch=2, x=FAKE, a_idx=FAKE, a_off=FAKE,
                n_gen=FAKE, a_total=10, a_max=5, gen_max=2, scores=None, score_layer=-1,
                workspace=FAKE, workspace_bytes=0)
    args.update(kw)
    L = binding.lib()
    return L.marche_step(C.byref(m), layers if layers is not None else _layers(m.n_layers),
                         C.byref(cache if cache is not None else _cache(m)), args["layer_begin"],
                         args["layer_end"], args["batch"], args["x"], args["a_idx"], args["a_off"],
                         args["n_gen"], args["a_total"], args["a_max"], args["gen_max"],
                         args["scores"], args["score_layer"], args["workspace"],
                         args["workspace_bytes"], None)


def test_status_strings():
    assert binding.status_string(0) == "MARCHE_OK"
    assert binding.status_string(4) == "MARCHE_ERR_WORKSPACE"
    assert binding.status_string(99) == "MARCHE_STATUS_UNKNOWN"


@pytest.mark.parametrize("kw,status,word", [
    (dict(head_dim=96, d_model=1536, n_heads=16), binding.MARCHE_ERR_UNSUPPORTED, "head_dim"),
    (dict(d_model=1000), binding.MARCHE_ERR_INVALID_ARG, "d_model"),
    (dict(dtype=7), binding.MARCHE_ERR_UNSUPPORTED, "dtype"),
    (dict(d_mlp=1000), binding.MARCHE_ERR_UNSUPPORTED, "d_mlp"),
    (dict(n_tokens=0), binding.MARCHE_ERR_INVALID_ARG, "n_tokens"),
    (dict(n_layers=0), binding.MARCHE_ERR_INVALID_ARG, "n_layers"),
])
def test_model_validation(kw, status, word):
    m = _model(**kw)
    assert _step(m) == status
    assert word in binding.last_error()


def test_step_argument_validation():
    m = _model()
    assert _step(m, layer_begin=1, layer_end=3) == binding.MARCHE_ERR_INVALID_ARG
    assert "layer range" in binding.last_error()
    assert _step(m, a_total=2 * 320 + 1) == binding.MARCHE_ERR_INVALID_ARG
    assert _step(m, a_max=400) == binding.MARCHE_ERR_INVALID_ARG
    assert _step(m, gen_max=6) == binding.MARCHE_ERR_INVALID_ARG
    assert _step(m, batch=3) == binding.MARCHE_ERR_INVALID_ARG  # cache holds 2 images
    assert _step(m, x=None) == binding.MARCHE_ERR_INVALID_ARG
    assert _step(m, scores=FAKE, score_layer=0, n_gen=None) == binding.MARCHE_ERR_INVALID_ARG
    bad = _layers(2)
    bad[1].w_o = None
    assert _step(m, layers=bad) == binding.MARCHE_ERR_INVALID_ARG
    assert "layers[1]" in binding.last_error()
    mism = _cache(m)
    mism.head_dim = 80
    assert _step(m, cache=mism) == binding.MARCHE_ERR_INVALID_ARG


def _step_images(m, first, batch, cache=None, **kw):
    args = dict(layer_begin=0, layer_end=m.n_layers, x=FAKE, a_idx=FAKE, a_off=FAKE, n_gen=FAKE,
                a_total=10, a_max=5, gen_max=2, scores=None, score_layer=-1, workspace=FAKE,
                workspace_bytes=0)
    args.update(kw)
    return binding.lib().marche_step_images(
        C.byref(m), _layers(m.n_layers), C.byref(cache if cache is not None else _cache(m, 4)),
        first, args["layer_begin"], args["layer_end"], batch, args["x"], args["a_idx"],
        args["a_off"], args["n_gen"], args["a_total"], args["a_max"], args["gen_max"],
        args["scores"], args["score_layer"], args["workspace"], args["workspace_bytes"], None)


def test_step_images_range_validation():
    m = _model()
    # images [first, first + batch) must lie inside the cache's 4 images
    for first, batch in ((-1, 2), (3, 2), (5, 0), (0, 5)):
        assert _step_images(m, first, batch) == binding.MARCHE_ERR_INVALID_ARG, (first, batch)
    assert "outside" in binding.last_error()
    # a valid range reaches the workspace check (nothing is launched)
    assert _step_images(m, 2, 2) == binding.MARCHE_ERR_WORKSPACE
    assert _step_images(m, 4, 0, a_total=0, a_max=0, gen_max=0) == binding.MARCHE_OK
    assert _step_images(m, 1, 2, layer_begin=1, layer_end=1) == binding.MARCHE_OK


def test_workspace_validation_and_size():
    m = _model()
    need = binding.workspace_bytes(m, 2, 10)
    # map + 2 * [M][D] bf16 + [M][F] bf16, each rounded up to 256 bytes
    assert need == 256 + 2 * 20480 + 81920
    assert _step(m, workspace_bytes=need - 1) == binding.MARCHE_ERR_WORKSPACE
    assert _step(m, workspace=None, workspace_bytes=need) == binding.MARCHE_ERR_WORKSPACE
    assert _step(m, workspace=FAKE + 8, workspace_bytes=need) == binding.MARCHE_ERR_INVALID_ARG
    # nothing to do: returns OK without touching memory
    assert _step(m, layer_begin=1, layer_end=1) == binding.MARCHE_OK
    assert _step(m, a_total=0, a_max=0, gen_max=0) == binding.MARCHE_OK


def test_select_refresh_validation():
    L = binding.lib()
    assert L.select_refresh(FAKE, 16, FAKE, FAKE, 2, 320, 321, FAKE, FAKE, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.select_refresh(FAKE, 0, FAKE, FAKE, 2, 320, 3, FAKE, FAKE, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.select_refresh(FAKE, 16, FAKE, FAKE, 2, 5000, 3, FAKE, FAKE, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.select_refresh(None, 16, FAKE, FAKE, 2, 320, 3, FAKE, FAKE, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.select_refresh(FAKE, 16, FAKE, FAKE, 2, 320, 0, FAKE, FAKE, None) == binding.MARCHE_OK
    assert L.select_refresh_ordered(FAKE, 16, FAKE, FAKE, 2, 320, 3, FAKE, FAKE, 2, None) == binding.MARCHE_ERR_INVALID_ARG
    assert "order" in binding.last_error()
    assert L.select_refresh_ordered(FAKE, 16, FAKE, FAKE, 2, 320, 0, FAKE, FAKE, 1, None) == binding.MARCHE_OK


def test_kv_cache_init_and_decoder_input_validation():
    L = binding.lib()
    m = _model()
    c = binding.KVCache()
    need = 2 * 3 * 16 * 320 * 64 * 2
    assert L.kv_cache_init(C.byref(c), C.byref(m), 3, FAKE, FAKE, need - 1, None, None, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.kv_cache_init(C.byref(c), C.byref(m), 3, FAKE, FAKE, need, FAKE, None, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.kv_cache_init(C.byref(c), C.byref(m), 3, FAKE + 2, FAKE, need, None, None, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.kv_cache_init(None, C.byref(m), 3, FAKE, FAKE, need, None, None, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.marche_decoder_input(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 320, 64, 1024, 257, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.marche_decoder_input(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 320, 400, 1024, 0, None) == binding.MARCHE_ERR_INVALID_ARG
    assert L.marche_decoder_input(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 320, 64, 1024, 0, None) == binding.MARCHE_OK


def test_profile_entry_bounds():
    binding.profile_reset()
    assert binding.lib().marche_profile_entry(-1, None, None, None, None, None) == binding.MARCHE_ERR_INVALID_ARG
    assert binding.profile_collect() == {}


def test_attention_segments_validation_and_workspace():
    L = binding.lib()
    bf16, f32 = binding.MARCHE_BF16, binding.MARCHE_F32
    two, cat = binding.MARCHE_ATTN_TWO_SEGMENT, binding.MARCHE_ATTN_CONCAT

    def call(mode=two, dtype=bf16, head_dim=64, n_query=32, n_a=32, n_c=256, batch=2, ws=None,
             ws_bytes=0, q=FAKE, k_c=FAKE):
        return L.marche_attention_segments(q, FAKE, n_query, FAKE, FAKE, n_a, k_c, k_c, n_c, batch,
                                           16, head_dim, dtype, mode, ws, ws_bytes, None)

    assert call(mode=2) == binding.MARCHE_ERR_INVALID_ARG
    assert "mode" in binding.last_error()
    assert call(dtype=f32) == binding.MARCHE_ERR_UNSUPPORTED
    assert call(head_dim=96) == binding.MARCHE_ERR_UNSUPPORTED
    assert call(n_query=0) == binding.MARCHE_ERR_INVALID_ARG
    assert call(n_a=0, n_c=0) == binding.MARCHE_ERR_INVALID_ARG
    assert call(n_c=-1) == binding.MARCHE_ERR_INVALID_ARG
    assert call(q=None) == binding.MARCHE_ERR_INVALID_ARG
    assert call(k_c=None) == binding.MARCHE_ERR_INVALID_ARG
    assert call(q=FAKE + 8) == binding.MARCHE_ERR_INVALID_ARG
    assert call(batch=0) == binding.MARCHE_OK
    need = binding.attention_workspace_bytes(2, 16, 64, 32, 256, bf16, cat)
    one = 2 * 16 * (32 + 256) * 64 * 2
    assert need == 2 * ((one + 255) // 256 * 256)
    assert binding.attention_workspace_bytes(2, 16, 64, 32, 256, bf16, two) == 0
    assert call(mode=cat) == binding.MARCHE_ERR_WORKSPACE
    assert call(mode=cat, ws=FAKE, ws_bytes=need - 1) == binding.MARCHE_ERR_WORKSPACE
    assert call(mode=cat, ws=FAKE + 16, ws_bytes=need) == binding.MARCHE_ERR_INVALID_ARG


def test_encoder_and_decoder_input_validation():
    L = binding.lib()
    f32, bf16 = binding.MARCHE_F32, binding.MARCHE_BF16

    def enc(batch=2, n_buf=4, n_img=32, n_known=8, d=256, c=16, x=FAKE, known=FAKE):
        return L.marche_encoder_input(x, FAKE, FAKE, FAKE, FAKE, FAKE, known, batch, n_buf, n_img,
                                      n_known, d, c, None)

    assert enc(n_known=33) == binding.MARCHE_ERR_INVALID_ARG
    assert enc(d=320) == binding.MARCHE_ERR_UNSUPPORTED
    assert enc(c=65) == binding.MARCHE_ERR_UNSUPPORTED
    assert enc(x=None) == binding.MARCHE_ERR_INVALID_ARG
    assert enc(known=None) == binding.MARCHE_ERR_INVALID_ARG
    assert enc(batch=0) == binding.MARCHE_OK  # nothing to do: no HIP call

    def e2d(dtype=bf16, n_known=8, d=256, ws=FAKE, ws_bytes=1 << 20, eps=1e-6, batch=2, rank=FAKE):
        return L.marche_encoder_to_decoder(FAKE, FAKE, FAKE, FAKE, eps, FAKE, FAKE, FAKE, FAKE, FAKE,
                                           rank, batch, 4, 32, n_known, d, dtype, ws, ws_bytes, None)

    assert e2d(dtype=5) == binding.MARCHE_ERR_UNSUPPORTED
    assert e2d(n_known=-1) == binding.MARCHE_ERR_INVALID_ARG
    assert e2d(d=100) == binding.MARCHE_ERR_UNSUPPORTED
    assert e2d(eps=0.0) == binding.MARCHE_ERR_INVALID_ARG
    assert e2d(rank=None) == binding.MARCHE_ERR_INVALID_ARG
    need = binding.encoder_to_decoder_workspace_bytes(2, 4, 8, 256, bf16)
    assert need == (2 * 12 * 256 * 2 + 255) // 256 * 256
    assert binding.encoder_to_decoder_workspace_bytes(2, 4, 8, 256, f32) == 2 * 12 * 256 * 4
    assert e2d(ws=None) == binding.MARCHE_ERR_WORKSPACE
    assert e2d(ws_bytes=need - 1) == binding.MARCHE_ERR_WORKSPACE
    assert e2d(ws=FAKE + 16) == binding.MARCHE_ERR_INVALID_ARG
    assert e2d(batch=0) == binding.MARCHE_OK


def test_diffusion_sample_validation_and_workspace():
    L = binding.lib()
    bf16 = binding.MARCHE_BF16
    wts = binding.HeadWeights(*([FAKE] * 16))

    def call(head=None, n_rows=10, n_steps=8, ws=FAKE, ws_bytes=1 << 30, tau=1.0, weights=wts,
             noise=FAKE, n_tokens=36, n_buf=4):
        hd = head or binding.make_head(256, 2, 16, 256, 256, bf16, 1e-6)
        return L.marche_diffusion_sample(C.byref(hd), C.byref(weights), FAKE, n_tokens, n_buf, FAKE,
                                         FAKE, 1e-6, FAKE, FAKE, FAKE, n_rows, noise, n_steps, tau,
                                         FAKE, ws, ws_bytes, None)

    for kw, status in [(dict(width=300), binding.MARCHE_ERR_UNSUPPORTED),
                       (dict(n_blocks=0), binding.MARCHE_ERR_UNSUPPORTED),
                       (dict(c_tok=65), binding.MARCHE_ERR_UNSUPPORTED),
                       (dict(d_cond=128), binding.MARCHE_ERR_UNSUPPORTED),
                       (dict(t_freq=96), binding.MARCHE_ERR_UNSUPPORTED),
                       (dict(dtype=7), binding.MARCHE_ERR_UNSUPPORTED),
                       (dict(ln_eps=0.0), binding.MARCHE_ERR_INVALID_ARG)]:
        h = dict(width=256, n_blocks=2, c_tok=16, d_cond=256, t_freq=256, dtype=bf16, ln_eps=1e-6)
        h.update(kw)
        assert call(head=binding.make_head(**h)) == status, kw
    assert call(n_steps=0) == binding.MARCHE_ERR_INVALID_ARG
    assert call(n_steps=10001) == binding.MARCHE_ERR_INVALID_ARG
    assert call(n_rows=-1) == binding.MARCHE_ERR_INVALID_ARG
    assert call(tau=-1.0) == binding.MARCHE_ERR_INVALID_ARG
    assert call(tau=float("nan")) == binding.MARCHE_ERR_INVALID_ARG
    assert call(n_buf=36) == binding.MARCHE_ERR_INVALID_ARG
    assert call(noise=None) == binding.MARCHE_ERR_INVALID_ARG
    assert call(weights=binding.HeadWeights(*([FAKE] * 15 + [None]))) == binding.MARCHE_ERR_INVALID_ARG
    assert call(n_rows=0) == binding.MARCHE_OK
    hd = binding.make_head(256, 2, 16, 256, 256, bf16, 1e-6)
    need = binding.diffusion_workspace_bytes(hd, 10, 8)
    a = lambda v: (v + 255) // 256 * 256
    W, M, T = 256, 10, 8
    assert need == (a(M * 256 * 2) + a(M * W * 4) + a(T * 256 * 2) + a(T * W * 2) + a(T * W * 4) +
                    a(M * W * 2) + a(M * 8 * W * 2) + a(M * W * 4) + 2 * a(M * W * 2) + a(M * W * 4) +
                    a(M * 16 * 4) + a(W * 16 * 4))
    assert call(ws=None) == binding.MARCHE_ERR_WORKSPACE
    assert call(ws_bytes=need - 1) == binding.MARCHE_ERR_WORKSPACE
    assert call(ws=FAKE + 64) == binding.MARCHE_ERR_INVALID_ARG


def test_layer_array_keeps_its_tensors_alive():
    """make_layers stores raw addresses; the array it returns holds the tensors,
    so dropping the caller's own references frees nothing (a freed weight's
    memory would be handed to the next allocation and read as weights)."""
    import gc
    import weakref

    import torch

    names = [n for n, _ in binding.Layer._fields_]
    params = [{n: torch.ones(4) for n in names} for _ in range(2)]
    probes = [weakref.ref(p[n]) for p in params for n in names]
    addrs = [p["w_qkv"].data_ptr() for p in params]
    arr = binding.make_layers(params)
    del params
    gc.collect()
    assert all(r() is not None for r in probes)
    assert [arr[i].w_qkv for i in range(2)] == addrs
    del arr
    gc.collect()
    assert all(r() is None for r in probes)


def test_step_noalloc_rejects_oversize_before_any_hip_call():
    """The no-allocation step refuses a step whose workspace would exceed the
    library-owned array, on the host (no GPU here), and its other checks are
    marche_step_images's."""
    m = _model()
    L = binding.lib()
    big = 6000  # rows: 6000 * (16 + 2*1024*2 + 4096*2) bytes > 64 MiB
    assert L.marche_step_workspace_bytes(C.byref(m), 20, big) > binding.SCRATCH_BYTES
    st = L.marche_step_images_noalloc(C.byref(m), _layers(m.n_layers), C.byref(_cache(m, 20)), 0,
                                      0, m.n_layers, 20, FAKE, FAKE, FAKE, FAKE, big, 320, 1, None,
                                      -1, None)
    assert st == binding.MARCHE_ERR_WORKSPACE
    assert "MARCHE_SCRATCH_BYTES" in binding.last_error()
    header = open(HEADER).read()
    assert "#define MARCHE_SCRATCH_BYTES ((size_t)64 << 20)" in header
    assert binding.SCRATCH_BYTES == 64 << 20
