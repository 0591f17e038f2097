"""Build and call the single-lane CPU replay of the step kernel's logic
(tests/emul).  Test-only: it exercises the kernel's algorithm (compressed
tree, interval marks, ordered candidate list, collector) on the CPU."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

import paper_2601_18999_amd as K

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "emul")
SRC = os.path.join(HERE, "kvr_emul.cpp")
LIB = os.path.join(HERE, "libkvr_emul.so")
CORE = os.path.join(os.path.dirname(HERE), "..", "paper_2601_18999_amd", "csrc", "kvr_core.h")


def build(sanitize: bool = False) -> str:
    deps = [SRC, os.path.join(HERE, "emul_wave.h"), CORE,
            os.path.join(os.path.dirname(CORE), "kvr_layout.h")]
    out = LIB if not sanitize else LIB.replace(".so", "_asan.so")
    if os.path.exists(out) and all(os.path.getmtime(out) >= os.path.getmtime(d) for d in deps):
        return out
    flags = ["-std=c++17", "-O1", "-g", "-ffp-contract=off", "-fPIC", "-shared", "-Wno-unknown-pragmas"]
    if sanitize:
        flags += ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"]
    # a private temporary name: parallel test workers may build at once
    tmp = f"{out}.{os.getpid()}.tmp"
    subprocess.check_call(["g++", *flags, "-o", tmp, SRC])
    os.replace(tmp, out)
    return out


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        _lib.emul_run.restype = ctypes.c_int
        _lib.emul_run.argtypes = [ctypes.POINTER(K.KvrConfig), ctypes.c_uint64] + [ctypes.c_void_p] * 9 + [ctypes.c_uint32]
        _lib.emul_pipe_unsafe.restype = ctypes.c_uint64
        _lib.emul_pipe_steps.restype = ctypes.c_uint64
        _lib.emul_draw_index.restype = ctypes.c_uint32
        _lib.emul_draw_index.argtypes = [ctypes.c_uint64, ctypes.c_uint32]
        _lib.emul_draw_index_decided.restype = ctypes.c_int
        _lib.emul_draw_index_decided.argtypes = [ctypes.c_uint64, ctypes.c_uint32]
    return _lib


def run(stream, R, W, B, all_hits=True, ws=None, ucap=8192, **cfg):
    c = K.kvr_config_default(R, W, B, max(1, stream.max_len), **cfg)
    n = stream.n
    tok = np.ascontiguousarray(stream.tokens, np.int32)
    off = np.ascontiguousarray(stream.offsets, np.uint64)
    arr = np.ascontiguousarray(stream.arrival_us, np.int64)
    ol = np.ascontiguousarray(stream.out_len, np.uint16)
    route = np.zeros((R, n), np.int32)
    hits = np.zeros((R, n), np.int32)
    ah = np.zeros((R, n, W), np.int32) if all_hits else None
    st = (K.KvrWorkerStats * (R * W))()
    rc = lib().emul_run(ctypes.byref(c), n, tok.ctypes.data, off.ctypes.data, arr.ctypes.data, ol.ctypes.data,
                        route.ctypes.data, hits.ctypes.data, ah.ctypes.data if ah is not None else None, st,
                        ws.ctypes.data if ws is not None else None, ucap)
    flat = K._stats_dicts(st, R * W)
    return {"rc": rc, "route": route, "hits": hits, "all_hits": ah,
            "workers": [flat[r * W:(r + 1) * W] for r in range(R)],
            "pipe_unsafe": int(lib().emul_pipe_unsafe()), "pipe_steps": int(lib().emul_pipe_steps())}
