"""Convenience wrapper: device buffers and batching around the C ABI.

``Simulator`` allocates the workspace with torch, uploads a stream (from
``workload``) to HBM once, and calls ``kvr_route_batch`` over consecutive
chunks of it.  Argument marshalling only.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

from . import (kvr_config_default, kvr_destroy, kvr_init_replicas, kvr_queries_done, kvr_route_batch,
               kvr_stats, kvr_workspace_size, kvr_check)


class DeviceStream:
    """A query stream resident in device memory (absolute offsets)."""

    def __init__(self, stream, device):
        import torch
        self.n = stream.n
        self.tokens = torch.from_numpy(np.ascontiguousarray(stream.tokens, dtype=np.int32)).to(device)
        self.offsets = torch.from_numpy(
            np.ascontiguousarray(stream.offsets, dtype=np.uint64).view(np.int64)).to(device)
        self.arrival = torch.from_numpy(np.ascontiguousarray(stream.arrival_us, dtype=np.int64)).to(device)
        self.out_len = torch.from_numpy(
            np.ascontiguousarray(stream.out_len, dtype=np.uint16).view(np.int16)).to(device)
        self.max_len = stream.max_len


class Simulator:
    def __init__(self, R: int, W: int, B: int, max_query_tokens: int, device: str = "cuda:0",
                 torch_stream=None, **cfg):
        import torch
        self.torch = torch
        self.device = torch.device(device)
        self.R, self.W, self.B = R, W, B
        self.cfg = kvr_config_default(R, W, B, max_query_tokens, **cfg)
        self.nbytes = kvr_workspace_size(self.cfg)
        with torch.cuda.device(self.device):
            self.stream = torch_stream or torch.cuda.current_stream(self.device)
            self.ws = torch.empty(self.nbytes, dtype=torch.uint8, device=self.device)
            self.ctx = kvr_init_replicas(self.cfg, self.ws.data_ptr(), self.nbytes, self.stream.cuda_stream)

    def upload(self, stream) -> DeviceStream:
        return DeviceStream(stream, self.device)

    def alloc_outputs(self, n: int, all_hits: bool = False) -> Dict[str, object]:
        t = self.torch
        out = {"route": t.empty((self.R, n), dtype=t.int32, device=self.device),
               "hits": t.empty((self.R, n), dtype=t.int32, device=self.device)}
        if all_hits:
            out["all_hits"] = t.empty((self.R, n, self.W), dtype=t.int32, device=self.device)
        return out

    def route(self, ds: DeviceStream, start: int, n: int, out: Optional[Dict[str, object]] = None,
              all_hits: bool = False) -> Dict[str, object]:
        """Route queries [start, start+n) of a device stream (one kvr_route_batch call)."""
        if out is None:
            out = self.alloc_outputs(n, all_hits)
        ah = out.get("all_hits")
        off = ds.offsets[start:start + n + 1]
        kvr_route_batch(self.ctx, n, ds.tokens.data_ptr(), off.data_ptr(),
                        ds.arrival[start:start + n].data_ptr(), ds.out_len[start:start + n].data_ptr(),
                        out["route"].data_ptr(), out["hits"].data_ptr(),
                        ah.data_ptr() if ah is not None else 0)
        return out

    def run(self, stream, batch: int = 0, all_hits: bool = False) -> Dict[str, np.ndarray]:
        """Route a whole host stream (uploading it), in batches of `batch`."""
        ds = self.upload(stream)
        n = stream.n
        batch = batch or n
        routes, hits, allh = [], [], []
        for s in range(0, n, batch):
            m = min(batch, n - s)
            o = self.route(ds, s, m, all_hits=all_hits)
            routes.append(o["route"])
            hits.append(o["hits"])
            if all_hits:
                allh.append(o["all_hits"])
        self.stream.synchronize()
        t = self.torch
        res = {"route": t.cat(routes, 1).cpu().numpy(), "hits": t.cat(hits, 1).cpu().numpy()}
        if all_hits:
            res["all_hits"] = t.cat(allh, 1).cpu().numpy()
        return res

    def stats(self, check: bool = True):
        return kvr_stats(self.ctx, self.R, self.W, check=check)

    def replica_stats(self, check: bool = True):
        """(per-replica records [R], per-worker records [R][W])."""
        return kvr_stats(self.ctx, self.R, self.W, check=check, with_replicas=True)

    def check(self):
        return kvr_check(self.ctx)

    @property
    def queries_done(self) -> int:
        return kvr_queries_done(self.ctx)

    def close(self):
        if getattr(self, "ctx", 0):
            kvr_destroy(self.ctx)
            self.ctx = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
