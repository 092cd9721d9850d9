"""ctypes binding of libmarche.so (include/marche.h).

Argument marshalling only: every function forwards to the C ABI with plain
pointers and sizes.  Tensors may be passed as torch tensors (their
``data_ptr()`` is used) or as integer addresses.  The library is loaded on
first use; if it has not been built, loading raises -- there is no other
implementation to fall back to.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
# MARCHE_LIB_PATH names another build of the same ABI (the sanitized host
# build the ABI tests run under); by default the library next to this file.
LIB_PATH = os.environ.get("MARCHE_LIB_PATH") or os.path.join(_HERE, "libmarche.so")

MARCHE_OK, MARCHE_ERR_INVALID_ARG, MARCHE_ERR_UNSUPPORTED, MARCHE_ERR_HIP, MARCHE_ERR_WORKSPACE = range(5)
MARCHE_F32, MARCHE_BF16 = 0, 1

MARCHE_SELECT_HIGHEST, MARCHE_SELECT_LOWEST = 0, 1
MARCHE_ATTN_TWO_SEGMENT, MARCHE_ATTN_CONCAT = 0, 1

EXPORTED = (
    "kv_cache_init", "marche_step_workspace_bytes", "marche_step", "marche_step_images",
    "marche_step_images_noalloc", "select_refresh",
    "select_refresh_ordered",
    "marche_decoder_input", "marche_attention_workspace_bytes", "marche_attention_segments",
    "marche_encoder_input", "marche_encoder_to_decoder_workspace_bytes",
    "marche_encoder_to_decoder", "marche_diffusion_workspace_bytes", "marche_diffusion_sample",
    "marche_status_string", "marche_last_error",
    "marche_profile_enable", "marche_profile_collect", "marche_profile_entry",
    "marche_profile_reset",
)


class Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("head_dim", C.c_int32), ("d_mlp", C.c_int32), ("n_tokens", C.c_int32),
                ("dtype", C.c_int32), ("ln_eps", C.c_float)]


class Layer(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                                          "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")]


class KVCache(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("n_layers", C.c_int32),
                ("batch", C.c_int32), ("n_heads", C.c_int32), ("n_tokens", C.c_int32),
                ("head_dim", C.c_int32), ("dtype", C.c_int32)]


class Head(C.Structure):
    _fields_ = [("width", C.c_int32), ("n_blocks", C.c_int32), ("c_tok", C.c_int32),
                ("d_cond", C.c_int32), ("t_freq", C.c_int32), ("dtype", C.c_int32),
                ("ln_eps", C.c_float)]


class HeadWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("w_t1", "b_t1", "w_t2", "b_t2", "w_c", "b_c", "w_in",
                                          "b_in", "w_ada", "b_ada", "w_1", "b_1", "w_2", "b_2",
                                          "w_out", "b_out")]


class MarcheError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run paper_2506_12035_amd.build.build()")
        L = C.CDLL(LIB_PATH)
        vp, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
        L.kv_cache_init.argtypes = [C.POINTER(KVCache), C.POINTER(Model), i32, vp, vp, sz, vp, vp, vp]
        L.marche_step_workspace_bytes.argtypes = [C.POINTER(Model), i32, i32]
        L.marche_step_workspace_bytes.restype = sz
        L.marche_step.argtypes = [C.POINTER(Model), C.POINTER(Layer), C.POINTER(KVCache), i32, i32,
                                  i32, vp, vp, vp, vp, i32, i32, i32, vp, i32, vp, sz, vp]
        L.marche_step_images.argtypes = [C.POINTER(Model), C.POINTER(Layer), C.POINTER(KVCache),
                                         i32, i32, i32, i32, vp, vp, vp, vp, i32, i32, i32, vp,
                                         i32, vp, sz, vp]
        L.marche_step_images_noalloc.argtypes = [C.POINTER(Model), C.POINTER(Layer),
                                                 C.POINTER(KVCache), i32, i32, i32, i32, vp, vp,
                                                 vp, vp, i32, i32, i32, vp, i32, vp]
        L.select_refresh.argtypes = [vp, i32, vp, vp, i32, i32, i32, vp, vp, vp]
        L.select_refresh_ordered.argtypes = [vp, i32, vp, vp, i32, i32, i32, vp, vp, i32, vp]
        L.marche_decoder_input.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, vp]
        L.marche_attention_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32, i32]
        L.marche_attention_workspace_bytes.restype = sz
        L.marche_attention_segments.argtypes = [vp, vp, i32, vp, vp, i32, vp, vp, i32, i32, i32,
                                                i32, i32, i32, vp, sz, vp]
        L.marche_encoder_input.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32,
                                           i32, vp]
        L.marche_encoder_to_decoder_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
        L.marche_encoder_to_decoder_workspace_bytes.restype = sz
        L.marche_encoder_to_decoder.argtypes = [vp, vp, vp, vp, C.c_float, vp, vp, vp, vp, vp, vp,
                                                i32, i32, i32, i32, i32, i32, vp, sz, vp]
        L.marche_diffusion_workspace_bytes.argtypes = [C.POINTER(Head), i32, i32]
        L.marche_diffusion_workspace_bytes.restype = sz
        L.marche_diffusion_sample.argtypes = [C.POINTER(Head), C.POINTER(HeadWeights), vp, i32,
                                              i32, vp, vp, C.c_float, vp, vp, vp, i32, vp, i32,
                                              C.c_float, vp, vp, sz, vp]
        L.marche_status_string.argtypes = [C.c_int]
        L.marche_status_string.restype = C.c_char_p
        L.marche_last_error.argtypes = []
        L.marche_last_error.restype = C.c_char_p
        L.marche_profile_enable.argtypes = [i32]
        L.marche_profile_collect.argtypes = []
        L.marche_profile_collect.restype = i32
        L.marche_profile_entry.argtypes = [i32, C.POINTER(C.c_char_p), C.POINTER(C.c_int64),
                                           C.POINTER(C.c_double), C.POINTER(C.c_double),
                                           C.POINTER(C.c_double)]
        L.marche_profile_reset.argtypes = []
        L.marche_profile_reset.restype = None
        for name in ("kv_cache_init", "marche_step", "marche_step_images",
                     "marche_step_images_noalloc", "select_refresh",
                     "select_refresh_ordered",
                     "marche_decoder_input", "marche_attention_segments",
                     "marche_encoder_input", "marche_encoder_to_decoder",
                     "marche_diffusion_sample", "marche_profile_enable", "marche_profile_entry"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().marche_status_string(s).decode()


def last_error() -> str:
    return lib().marche_last_error().decode()


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _check(status: int) -> None:
    if status != MARCHE_OK:
        raise MarcheError(status, last_error())


def _stream(stream) -> Optional[int]:
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_model(n_layers, d_model, n_heads, head_dim, d_mlp, n_tokens, dtype, ln_eps) -> Model:
    return Model(n_layers, d_model, n_heads, head_dim, d_mlp, n_tokens, dtype, ln_eps)


def make_layers(params: Sequence[dict]):
    """ctypes array of Layer from dicts of device tensors / addresses.

    The array holds raw device addresses, so it keeps the dicts (and with them
    the tensors) alive for as long as it lives: a caller that drops its own
    references cannot have the weights freed and their memory reused under a
    later step."""
    arr = (Layer * len(params))()
    for i, p in enumerate(params):
        for name, _ in Layer._fields_:
            setattr(arr[i], name, _ptr(p[name]))
    arr._owners = [dict(p) for p in params]
    return arr


def kv_cache_init(model: Model, batch: int, k_buf, v_buf, bytes_each: int, k_init=None,
                  v_init=None, stream=None) -> KVCache:
    cache = KVCache()
    _check(lib().kv_cache_init(C.byref(cache), C.byref(model), batch, _ptr(k_buf), _ptr(v_buf),
                               bytes_each, _ptr(k_init), _ptr(v_init), _stream(stream)))
    cache._owners = (k_buf, v_buf)  # the handle points into these buffers: keep them alive
    return cache


def workspace_bytes(model: Model, batch: int, a_total: int) -> int:
    return lib().marche_step_workspace_bytes(C.byref(model), batch, a_total)


def marche_step(model: Model, layers, cache: KVCache, layer_begin: int, layer_end: int, batch: int,
                x, a_idx, a_off, n_gen, a_total: int, a_max: int, gen_max: int, scores=None,
                score_layer: int = -1, workspace=None, workspace_bytes: int = 0,
                stream=None) -> None:
    _check(lib().marche_step(C.byref(model), layers, C.byref(cache), layer_begin, layer_end, batch,
                             _ptr(x), _ptr(a_idx), _ptr(a_off), _ptr(n_gen), a_total, a_max,
                             gen_max, _ptr(scores), score_layer, _ptr(workspace), workspace_bytes,
                             _stream(stream)))


def marche_step_images(model: Model, layers, cache: KVCache, first_image: int, layer_begin: int,
                       layer_end: int, batch: int, x, a_idx, a_off, n_gen, a_total: int,
                       a_max: int, gen_max: int, scores=None, score_layer: int = -1,
                       workspace=None, workspace_bytes: int = 0, stream=None) -> None:
    _check(lib().marche_step_images(C.byref(model), layers, C.byref(cache), first_image,
                                    layer_begin, layer_end, batch, _ptr(x), _ptr(a_idx),
                                    _ptr(a_off), _ptr(n_gen), a_total, a_max, gen_max,
                                    _ptr(scores), score_layer, _ptr(workspace), workspace_bytes,
                                    _stream(stream)))


# Bytes of the library-owned workspace of marche_step_images_noalloc
# (MARCHE_SCRATCH_BYTES in include/marche.h).
SCRATCH_BYTES = 64 << 20


def marche_step_images_noalloc(model: Model, layers, cache: KVCache, first_image: int,
                               layer_begin: int, layer_end: int, batch: int, x, a_idx, a_off,
                               n_gen, a_total: int, a_max: int, gen_max: int, scores=None,
                               score_layer: int = -1, stream=None) -> None:
    _check(lib().marche_step_images_noalloc(C.byref(model), layers, C.byref(cache), first_image,
                                            layer_begin, layer_end, batch, _ptr(x), _ptr(a_idx),
                                            _ptr(a_off), _ptr(n_gen), a_total, a_max, gen_max,
                                            _ptr(scores), score_layer, _stream(stream)))


def select_refresh(scores, n_parts: int, excl_idx, excl_off, batch: int, n_tokens: int, k: int,
                   out_idx, out_off, stream=None, lowest: bool = False) -> None:
    order = MARCHE_SELECT_LOWEST if lowest else MARCHE_SELECT_HIGHEST
    _check(lib().select_refresh_ordered(_ptr(scores), n_parts, _ptr(excl_idx), _ptr(excl_off),
                                        batch, n_tokens, k, _ptr(out_idx), _ptr(out_off), order,
                                        _stream(stream)))


def decoder_input(x, cls, value, mask, pos, rank, batch: int, n_tokens: int, n_buf: int,
                  d_model: int, n_known: int, stream=None) -> None:
    _check(lib().marche_decoder_input(_ptr(x), _ptr(cls), _ptr(value), _ptr(mask), _ptr(pos),
                                      _ptr(rank), batch, n_tokens, n_buf, d_model, n_known,
                                      _stream(stream)))


def attention_workspace_bytes(batch: int, n_heads: int, head_dim: int, n_a: int, n_c: int,
                              dtype: int, mode: int) -> int:
    return lib().marche_attention_workspace_bytes(batch, n_heads, head_dim, n_a, n_c, dtype, mode)


def attention_segments(q, o, n_query: int, k_a, v_a, n_a: int, k_c, v_c, n_c: int, batch: int,
                       n_heads: int, head_dim: int, dtype: int, mode: int, workspace=None,
                       workspace_bytes: int = 0, stream=None) -> None:
    _check(lib().marche_attention_segments(_ptr(q), _ptr(o), n_query, _ptr(k_a), _ptr(v_a), n_a,
                                           _ptr(k_c), _ptr(v_c), n_c, batch, n_heads, head_dim,
                                           dtype, mode, _ptr(workspace), workspace_bytes,
                                           _stream(stream)))


def encoder_input(x_enc, cls, tok, w_z, b_z, pe_enc, known, batch: int, n_buf: int, n_img: int,
                  n_known: int, d_model: int, c_tok: int, stream=None) -> None:
    _check(lib().marche_encoder_input(_ptr(x_enc), _ptr(cls), _ptr(tok), _ptr(w_z), _ptr(b_z),
                                      _ptr(pe_enc), _ptr(known), batch, n_buf, n_img, n_known,
                                      d_model, c_tok, _stream(stream)))


def encoder_to_decoder_workspace_bytes(batch: int, n_buf: int, n_known: int, d_model: int,
                                       dtype: int) -> int:
    return lib().marche_encoder_to_decoder_workspace_bytes(batch, n_buf, n_known, d_model, dtype)


def encoder_to_decoder(x_dec, x_enc, ln_g, ln_b, ln_eps: float, w_de, b_de, mask, pe_dec, known,
                       rank, batch: int, n_buf: int, n_img: int, n_known: int, d_model: int,
                       dtype: int, workspace=None, workspace_bytes: int = 0, stream=None) -> None:
    _check(lib().marche_encoder_to_decoder(_ptr(x_dec), _ptr(x_enc), _ptr(ln_g), _ptr(ln_b), ln_eps,
                                           _ptr(w_de), _ptr(b_de), _ptr(mask), _ptr(pe_dec),
                                           _ptr(known), _ptr(rank), batch, n_buf, n_img, n_known,
                                           d_model, dtype, _ptr(workspace), workspace_bytes,
                                           _stream(stream)))


def make_head(width, n_blocks, c_tok, d_cond, t_freq, dtype, ln_eps) -> Head:
    return Head(width, n_blocks, c_tok, d_cond, t_freq, dtype, ln_eps)


def make_head_weights(p: dict) -> HeadWeights:
    w = HeadWeights()
    for name, _ in HeadWeights._fields_:
        setattr(w, name, _ptr(p[name]))
    return w


def diffusion_workspace_bytes(head: Head, n_rows: int, n_steps: int) -> int:
    return lib().marche_diffusion_workspace_bytes(C.byref(head), n_rows, n_steps)


def diffusion_sample(head: Head, weights: HeadWeights, x_dec, n_tokens: int, n_buf: int, dec_ln_g,
                     dec_ln_b, dec_ln_eps: float, pe_diff, rows, out_rows, n_rows: int, noise,
                     n_steps: int, temperature: float, tok_out, workspace=None,
                     workspace_bytes: int = 0, stream=None) -> None:
    _check(lib().marche_diffusion_sample(C.byref(head), C.byref(weights), _ptr(x_dec), n_tokens,
                                         n_buf, _ptr(dec_ln_g), _ptr(dec_ln_b), dec_ln_eps,
                                         _ptr(pe_diff), _ptr(rows), _ptr(out_rows), n_rows,
                                         _ptr(noise), n_steps, temperature, _ptr(tok_out),
                                         _ptr(workspace), workspace_bytes, _stream(stream)))


def profile_enable(on: bool) -> None:
    _check(lib().marche_profile_enable(1 if on else 0))


def profile_reset() -> None:
    lib().marche_profile_reset()


def profile_collect() -> dict:
    """{kernel class: {launches, ms, flops, bytes}} for classes with launches."""
    L = lib()
    n = L.marche_profile_collect()
    out = {}
    for i in range(n):
        name = C.c_char_p()
        la, ms, fl, by = C.c_int64(), C.c_double(), C.c_double(), C.c_double()
        _check(L.marche_profile_entry(i, C.byref(name), C.byref(la), C.byref(ms), C.byref(fl),
                                      C.byref(by)))
        if la.value:
            out[name.value.decode()] = {"launches": la.value, "ms": ms.value, "flops": fl.value,
                                        "bytes": by.value}
    return out
