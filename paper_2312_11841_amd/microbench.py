"""Roofline microbenchmarks (libmixrt_microbench.so): achievable gather rate by
working-set size, streaming-copy and streaming-read bandwidth and fp16 MFMA
throughput on the
current GPU.  These calibrate the rendering kernel's measured bounds; they
are not part of the rendering path."""
from __future__ import annotations

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmixrt_microbench.so")
WORK_WORDS = 2560   # MIXRT_MB_WORK_WORDS: the replay's work counters
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build with paper_2312_11841_amd/build.py")
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        L.mixrt_mb_gather.argtypes = [P, C.c_uint64, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                      P, P]
        L.mixrt_mb_copy.argtypes = [P, P, C.c_uint64, C.c_int, P]
        L.mixrt_mb_gather_lines.argtypes = [P, C.c_uint64, C.c_int, C.c_int, C.c_int, C.c_int,
                                            C.c_int, P, P]
        L.mixrt_mb_gather_lines.restype = C.c_int
        L.mixrt_mb_read.argtypes = [P, C.c_uint64, C.c_int, P, P]
        L.mixrt_mb_mfma.argtypes = [C.c_int, C.c_int, P, P]
        L.mixrt_mb_rowstream.argtypes = [P, P, C.c_int64, C.c_int, C.c_int, P]
        L.mixrt_mb_rowstream.restype = C.c_int
        I32 = C.c_int32
        L.mixrt_mb_gather_replay.argtypes = [P, P, I32, I32, I32, I32, P, I32, I32, I32, P, I32,
                                             I32, I32, I32, I32, I32, P, P, P]
        L.mixrt_mb_gather_replay.restype = C.c_int
        IP = C.POINTER(C.c_int)
        L.mixrt_mb_device_info.argtypes = [C.c_int, IP, IP, IP, IP, C.c_char_p, C.c_int]
        for f in (L.mixrt_mb_gather, L.mixrt_mb_copy, L.mixrt_mb_read, L.mixrt_mb_mfma,
                  L.mixrt_mb_device_info):
            f.restype = C.c_int
        _lib = L
    return _lib


def _timed(launch, reps=5):
    import torch
    s = torch.cuda.current_stream()
    launch(s)  # warm
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(s)
    for _ in range(reps):
        launch(s)
    b.record(s)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps * 1e-3


def _check(rc):
    if rc != 0:
        raise RuntimeError(f"microbenchmark launch failed: hipError {rc}")


def gather(table_bytes: int, width: int = 4, pattern: int = 0, iters: int = 64,
           blocks: int | None = None):
    """Random (pattern 0) or coalesced (pattern 1) gathers; returns rates."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = blocks or cus * 8
    table = torch.randint(0, 2 ** 31, (table_bytes // 4,), dtype=torch.int32, device="cuda")
    sink = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    nl = 8

    def launch(s):
        _check(lib().mixrt_mb_gather(table.data_ptr(), table_bytes, width, nl, iters, pattern,
                                     blocks, sink.data_ptr(), s.cuda_stream))

    t = _timed(launch)
    lane_loads = blocks * 256 * iters * nl
    wave_instr = lane_loads / 64
    return {"table_bytes": table_bytes, "width": width, "pattern": pattern,
            "seconds": t, "lane_loads_per_s": lane_loads / t,
            "useful_GBps": lane_loads * width / t / 1e9,
            "wave_instr_per_s": wave_instr / t,
            "ns_per_wave_instr_per_cu": t * 1e9 * cus / wave_instr}


def gather_lines(table_bytes: int, width: int, lines: int, adjacent: bool,
                 blocks_per_cu: int = 4, iters: int = 256):
    """Cycles per gather instruction per CU (at the 2.4 GHz peak clock) when
    each instruction's 64 lanes touch `lines` distinct 128-byte lines
    (mixrt_mb_gather_lines)."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = blocks_per_cu * cus
    t = torch.randint(0, 2**31 - 1, (table_bytes // 4,), dtype=torch.int32, device="cuda")
    sink = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")

    def launch(s):
        _check(lib().mixrt_mb_gather_lines(t.data_ptr(), table_bytes, width, lines,
                                           int(bool(adjacent)), iters, blocks, sink.data_ptr(),
                                           s.cuda_stream))
    sec = _timed(launch, 10)
    instr_per_cu = blocks * 4 * iters * 8 / cus
    return sec * 2.4e9 / instr_per_cu


def copy(bytes_: int = 1 << 30, blocks: int | None = None):
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = blocks or cus * 8
    src = torch.empty(bytes_, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)

    def launch(s):
        _check(lib().mixrt_mb_copy(src.data_ptr(), dst.data_ptr(), bytes_, blocks, s.cuda_stream))

    t = _timed(launch)
    return {"bytes": bytes_, "blocks": blocks, "seconds": t, "GBps": 2 * bytes_ / t / 1e9}


def read(bytes_: int = 1 << 30, blocks: int | None = None):
    """Streaming read of bytes_; returns the read bandwidth."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = blocks or cus * 8
    src = torch.empty(bytes_, dtype=torch.uint8, device="cuda").fill_(1)
    sink = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")

    def launch(s):
        _check(lib().mixrt_mb_read(src.data_ptr(), bytes_, blocks, sink.data_ptr(),
                                   s.cuda_stream))

    t = _timed(launch)
    return {"bytes": bytes_, "blocks": blocks, "seconds": t, "GBps": bytes_ / t / 1e9}


def mfma(iters: int = 4096, blocks: int | None = None):
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = blocks or cus * 8
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")

    def launch(s):
        _check(lib().mixrt_mb_mfma(iters, blocks, out.data_ptr(), s.cuda_stream))

    t = _timed(launch)
    flops = blocks * 4 * iters * 8 * (2 * 16 * 16 * 32)
    return {"seconds": t, "TFLOPs": flops / t / 1e12}


def device_info(device: int = 0) -> dict:
    """Clock rates, CU count, L2 size and architecture of a HIP device."""
    clk, mclk, cus, l2 = C.c_int(), C.c_int(), C.c_int(), C.c_int()
    arch = C.create_string_buffer(64)
    _check(lib().mixrt_mb_device_info(device, C.byref(clk), C.byref(mclk), C.byref(cus),
                                      C.byref(l2), arch, 64))
    return {"clock_MHz": clk.value // 1000, "mem_clock_MHz": mclk.value // 1000,
            "compute_units": cus.value, "l2_bytes": l2.value, "arch": arch.value.decode()}


def gather_replay(x, hit, views: int, W: int, H: int, K: int, table, N, tile_stripe: int,
                  blocks_list, reps: int = 20, chunk: int = 0, block_from=None,
                  hash_batch: int = 2, claims: bool = True):
    """The frame's hash-grid loads replayed in the render kernel's order
    (mixrt_mb_gather_replay): for each grid size in blocks_list, the mean time
    of the loads (mode 0) and of their address arithmetic alone (mode 1).
    x: device float [rays][K][3] and hit: device int32 [rays] from the
    frame's ray setup; table: the device hash table [L][T][F]; N: level
    resolutions; chunk: the render's samples per ray per round (0: the tile
    path); block_from: the render's first level of 16-byte block gathers
    (None: none); hash_batch: its hashed levels per batch of gathers;
    claims: whether the waves claim their last runs from work counters (the
    plan's claims) or take every run in the fixed order.
    Returns per-grid-size times and the fastest."""
    import numpy as np
    import torch
    L_, T, F = (int(n) for n in table.shape)
    eb = F * table.element_size()
    Nh = np.ascontiguousarray(np.asarray(N, np.int32))
    assert x.is_cuda and hit.is_cuda and table.is_cuda and x.is_contiguous()
    assert x.numel() == views * H * W * K * 3 and hit.numel() == views * H * W
    assert Nh.size == L_ and T & (T - 1) == 0
    bf = L_ if block_from is None else int(block_from)
    rows = []
    work = torch.zeros(WORK_WORDS, dtype=torch.int32, device=x.device)
    for blocks in blocks_list:
        sink = torch.empty(int(blocks) * 256, dtype=torch.int32, device=x.device)
        res = {"blocks": int(blocks)}
        for mode, name in ((0, "ms"), (1, "address_only_ms")):
            def launch(s, mode=mode):
                _check(lib().mixrt_mb_gather_replay(
                    x.data_ptr(), hit.data_ptr(), views, W, H, K, table.data_ptr(), L_,
                    T.bit_length() - 1, eb, Nh.ctypes.data, int(tile_stripe), int(chunk), bf,
                    int(hash_batch), mode, int(blocks), work.data_ptr() if claims else None,
                    sink.data_ptr(), s.cuda_stream))
            for _ in range(3):
                launch(torch.cuda.current_stream())
            res[name] = _timed(launch, reps) * 1e3
        rows.append(res)
    best = min(rows, key=lambda r: r["ms"])
    return {"by_blocks": rows, "best": best}


def rowstream(rows: int, in_bytes: int = 96, blocks_list=None, reps: int = 20):
    """The MLP stage's memory pattern alone (mixrt_mb_rowstream): rows of
    in_bytes read, 16 bytes per row written.  Returns the fastest of the
    grid sizes tried, as bytes moved per second."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    rows -= rows % 64
    src = torch.empty(rows * in_bytes // 4, dtype=torch.int32, device="cuda")
    src.random_()
    dst = torch.empty(rows * 4, dtype=torch.int32, device="cuda")
    best = None
    for k in (blocks_list or (1, 2, 3, 4, 6, 8)):
        blocks = int(k * cus)

        def launch(s):
            _check(lib().mixrt_mb_rowstream(src.data_ptr(), dst.data_ptr(), rows, in_bytes,
                                            blocks, s.cuda_stream))
        t = _timed(launch, reps)
        r = {"blocks": blocks, "seconds": t, "GBps": rows * (in_bytes + 16) / t / 1e9}
        if best is None or r["GBps"] > best["GBps"]:
            best = r
    return {"rows": rows, "in_bytes": in_bytes, **best}
