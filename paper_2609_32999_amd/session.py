"""Device buffers for one attention layer of the composed-prefill path.

PyTorch provides device memory and streams only; every step of the path runs
in libtsr's kernels through the C ABI.  A Session owns, for one layer shape:

* the pool arena     [n_pool_pages][H_kv][B][d] for K (pre-RoPE) and V, in
                     device memory or, for the host tier, in pinned host
                     memory that the kernels read and write over the bus;
* the request arena  [n_req_pages][H_kv][B][d] for the assembled K and V;
* the RoPE table     built once per model by tsr_rope_table_init;
* for e4m3 pools, page scales [n_layers][pages][2] fp32 ({K, V}) for both
  arenas.

Plans (one per batch of requests) own their device workspace.
"""
from __future__ import annotations

import torch

from . import _binding as B

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16, "e4m3": torch.uint8}


def _require_device():
    if not torch.cuda.is_available():
        raise RuntimeError("libtsr needs a ROCm GPU; none is visible")


def _host_device_pointer(t: torch.Tensor) -> int:
    """Device-visible address of a pinned host tensor (hipHostGetDevicePointer
    on the HIP runtime torch has loaded)."""
    import ctypes
    if not t.is_pinned():
        raise RuntimeError("host-tier pools must be pinned host memory")
    hip = ctypes.CDLL("libamdhip64.so.7")
    dptr = ctypes.c_void_p()
    err = hip.hipHostGetDevicePointer(ctypes.byref(dptr), ctypes.c_void_p(t.data_ptr()), 0)
    if err != 0 or not dptr.value:
        raise RuntimeError(f"hipHostGetDevicePointer failed ({err})")
    return int(dptr.value)


class Session:
    def __init__(self, shape, n_pool_pages: int, n_req_pages: int,
                 device: str = "cuda", n_layers: int = 1, stream=None, pool: str = "device"):
        """`shape` has n_q_heads, n_kv_heads, head_dim, page_size, kv_dtype,
        act_dtype, rope_theta, max_position (workloads.ModelShape).  `pool`
        is "device" (HBM) or "host" (pinned host memory: the host tier)."""
        _require_device()
        B.lib()
        self.shape = shape
        self.model = B.make_model(shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                                  shape.page_size, shape.kv_dtype, shape.act_dtype,
                                  shape.rope_theta, shape.max_position)
        if shape.kv_dtype not in TORCH_DTYPE:
            raise B.TsrError(B.TSR_ERR_UNSUPPORTED, f"kv dtype {shape.kv_dtype}")
        self.device = torch.device(device)
        self.kv_dtype = TORCH_DTYPE[shape.kv_dtype]
        self.act_dtype = TORCH_DTYPE[shape.act_dtype]
        if shape.act_dtype == "e4m3":
            raise B.TsrError(B.TSR_ERR_UNSUPPORTED, "activations cannot be e4m3")
        self.n_layers = n_layers
        self.n_pool_pages = n_pool_pages
        self.n_req_pages = n_req_pages
        page = (shape.n_kv_heads, shape.page_size, shape.head_dim)
        if pool not in ("device", "host"):
            raise ValueError(f"pool must be 'device' or 'host', not {pool!r}")
        self.pool_tier = pool
        pool_dev = dict(device=self.device) if pool == "device" else dict(pin_memory=True)
        # K and V in one allocation, [K|V][layer][page]: every (K|V, layer)
        # slab sits a whole arena after the previous one, so one strided copy
        # can move a run of pages for K, V and every layer at once
        self.pool_kv = torch.empty((2, n_layers, n_pool_pages, *page), dtype=self.kv_dtype,
                                   **pool_dev)
        self.pool_k, self.pool_v = self.pool_kv[0], self.pool_kv[1]
        self.req_k = torch.empty((n_layers, n_req_pages, *page), dtype=self.kv_dtype,
                                 device=self.device)
        self.req_v = torch.empty_like(self.req_k)
        self.e4m3 = shape.kv_dtype == "e4m3"
        self.pool_scale = self.req_scale = None
        if self.e4m3:
            self.pool_scale = torch.empty((n_layers, n_pool_pages, 2), dtype=torch.float32,
                                          **pool_dev)
            self.req_scale = torch.empty((n_layers, n_req_pages, 2), dtype=torch.float32,
                                         device=self.device)
        # addresses the kernels use for the pool arenas
        self._pool_base = {}
        kv_base = (self.pool_kv.data_ptr() if pool == "device"
                   else _host_device_pointer(self.pool_kv))
        self._pool_base["pool_k"] = kv_base
        self._pool_base["pool_v"] = kv_base + self.pool_k.nbytes
        if self.pool_scale is not None:
            self._pool_base["pool_scale"] = (self.pool_scale.data_ptr() if pool == "device"
                                             else _host_device_pointer(self.pool_scale))
        nbytes = B.tsr_rope_table_bytes(self.model)
        if nbytes == 0:
            raise B.TsrError(B.TSR_ERR_INVALID_ARG, B.tsr_last_error())
        self.rope = torch.empty(nbytes // 4, dtype=torch.float32, device=self.device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        B.tsr_rope_table_init(self.model, self.rope, nbytes, self.stream)

    # ------------------------------------------------------------- plans
    def plan(self, requests, stream=None, alias_v: bool = False, alias_k: bool = False,
             split_tiles: int = 0, attn_kernel: int = 0):
        """Validate and upload a batch's plan; `alias_v` selects V aliasing
        (attention reads V of whole gathered pages from the pool), `alias_k`
        K rotated on load (attention reads their pre-RoPE K from the pool),
        `split_tiles` the key-range split of long attention items (0
        automatic, > 0 the most 32-key tiles an item keeps, -1 never),
        `attn_kernel` the bf16 attention kernel (0 automatic, 1 pipelined,
        2 row-block under its rule, 3 / 4 row-block with three / one row
        blocks)."""
        batch = B.RequestBatch(requests)
        ws_bytes = B.tsr_plan_workspace_size(self.model, batch, self.n_pool_pages,
                                             self.n_req_pages, alias_v, alias_k, split_tiles,
                                             attn_kernel)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=self.device)
        plan = B.tsr_plan_create(self.model, batch, self.n_pool_pages, self.n_req_pages,
                                 self.rope, ws, ws_bytes, stream or self.stream,
                                 alias_v=alias_v, alias_k=alias_k, split_tiles=split_tiles,
                                 attn_kernel=attn_kernel)
        plan.workspace = ws     # keep the workspace alive with the plan
        plan.batch = batch
        return plan

    def plan_static(self, requests, stream=None, alias_v: bool = False,
                    alias_k: bool = False, split_tiles: int = 0, attn_kernel: int = 0):
        """A plan in the library's own device plan area (no workspace is
        allocated); a later static plan on this device supersedes it."""
        batch = B.RequestBatch(requests)
        plan = B.tsr_plan_create_static(self.model, batch, self.n_pool_pages,
                                        self.n_req_pages, self.rope, stream or self.stream,
                                        alias_v=alias_v, alias_k=alias_k,
                                        split_tiles=split_tiles, attn_kernel=attn_kernel)
        plan.batch = batch
        return plan

    # ---------------------------------------------------------- hot path
    def compose(self, plan, layer: int | None = None, stream=None):
        """Compose one layer (default 0), or all layers when layer == 'all'."""
        s = stream or self.stream
        if layer == "all":
            B.tsr_compose_kv(plan, self._pk(0), self._pv(0), self._ps(0), self.req_k,
                             self.req_v, self.req_scale, self.n_layers,
                             self.pool_k[0].nbytes if self.n_layers > 1 else 0,
                             self.req_k[0].nbytes if self.n_layers > 1 else 0, s)
            return
        li = layer or 0
        B.tsr_compose_kv(plan, self._pk(li), self._pv(li), self._ps(li), self.req_k[li],
                         self.req_v[li], self._rs(li), 1, 0, 0, s)

    # kernel-visible addresses of one layer of the pool arenas
    def _pool_addr(self, name, layer):
        t = getattr(self, name)
        return self._pool_base[name] + layer * t[0].nbytes

    def _pk(self, layer):
        return self._pool_addr("pool_k", layer)

    def _pv(self, layer):
        return self._pool_addr("pool_v", layer)

    def _ps(self, layer):
        return self._pool_addr("pool_scale", layer) if self.e4m3 else None

    def _rs(self, layer):
        return self.req_scale[layer] if self.e4m3 else None

    def new_outputs(self, plan, with_lse: bool = True):
        T = plan.num_compute_tokens
        out = torch.empty((T, self.shape.n_q_heads, self.shape.head_dim),
                          dtype=self.act_dtype, device=self.device)
        lse = (torch.empty((T, self.shape.n_q_heads), dtype=torch.float32,
                           device=self.device) if with_lse else None)
        return out, lse

    def prefill_attn(self, plan, q, k, v, out, lse=None, layer: int = 0, stream=None):
        if getattr(plan, "alias_v", False) or getattr(plan, "alias_k", False):
            # append, then attention with pool K / V
            self.append(plan, k, v, layer=layer, stream=stream)
            self.attn(plan, q, out, lse, layer=layer, stream=stream)
            return
        B.tsr_prefill_attn(plan, q, k, v, self.req_k[layer], self.req_v[layer],
                           self._rs(layer), out, lse, stream or self.stream)

    def append(self, plan, k, v, layer: int = 0, stream=None):
        B.tsr_append_kv(plan, k, v, self.req_k[layer], self.req_v[layer], self._rs(layer),
                        stream or self.stream)

    def assemble(self, plan, k, v, layer: int = 0, stream=None):
        """compose + append of one layer in one launch (same results)."""
        B.tsr_assemble_kv(plan, self._pk(layer), self._pv(layer), self._ps(layer), k, v,
                          self.req_k[layer], self.req_v[layer], self._rs(layer),
                          stream or self.stream)

    def attn(self, plan, q, out, lse=None, layer: int = 0, stream=None, part: int = 0):
        """Attention over the assembled pages; `part` selects all items
        (TSR_ATTN_ALL) or the items before / after compose."""
        av, ak = getattr(plan, "alias_v", False), getattr(plan, "alias_k", False)
        if av or ak:
            B.tsr_attn_aliased(plan, part, q, self.req_k[layer], self.req_v[layer],
                               self._pk(layer) if ak else None,
                               self._pv(layer) if av else None, out, lse,
                               stream or self.stream)
            return
        B.tsr_attn_part(plan, part, q, self.req_k[layer], self.req_v[layer], self._rs(layer),
                        out, lse, stream or self.stream)

    def retain(self, plan, k, v, layer: int = 0, stream=None):
        B.tsr_retain_kv(plan, k, v, self._pk(layer), self._pv(layer), self._ps(layer),
                        stream or self.stream)
