"""Python face of the C ABI: a net of layers, profiling, routine-path
selection and inference.  PyTorch is used only to hold device tensors and to
name the stream; all computation happens in libsoftneuro.so.
"""

from __future__ import annotations

import ctypes
import json

import numpy as np

from . import native as N

_STORAGE = {N.F32: np.float32, N.F16: np.float16, N.BF16: np.uint16}


def _stream_ptr(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


class Graph:
    """A net (Sec. III-B of the paper) with its routine set and selected path.

    ``device=-1`` makes a host-only graph: only cost-table import, selection
    and queries work (no weights are uploaded)."""

    def __init__(self, dtype, n, c, h, w, device=0, layouts=None, algos=None, params=True, dtypes=None,
                 ws_limit=None):
        self.lib = N.lib()
        self.dtype = N.DTYPE[dtype] if isinstance(dtype, str) else dtype
        self.dtype_name = {v: k for k, v in N.DTYPE.items()}[self.dtype]
        self.device = device
        p = ctypes.c_void_p()
        N.check(self.lib.sn_graph_create(self.dtype, n, c, h, w, device, ctypes.byref(p)))
        self._g = p
        if layouts is not None:
            mask = sum(1 << N.LAYOUT[l] if isinstance(l, str) else 1 << l for l in layouts)
            self.set_option(N.OPT_LAYOUTS, mask)
        if algos is not None:
            mask = sum(1 << N.ALGO[a] if isinstance(a, str) else 1 << a for a in algos)
            self.set_option(N.OPT_ALGOS, mask)
        if not params:
            self.set_option(N.OPT_PARAMS, 0)
        if dtypes is not None:
            mask = sum(1 << (N.DTYPE[d] if isinstance(d, str) else d) for d in dtypes)
            self.set_option(N.OPT_DTYPES, mask)
        if ws_limit is not None:
            self.set_option(N.OPT_WS_LIMIT, ws_limit)
        self.in_shape = (n, c, h, w)
        self.in_shapes = [self.in_shape]

    # ---------------------------------------------------------------- lifetime
    def close(self):
        if getattr(self, "_g", None):
            self.lib.sn_graph_destroy(self._g)
            self._g = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def set_option(self, opt, value):
        N.check(self.lib.sn_set_option(self._g, opt, int(value)))

    # ---------------------------------------------------------------- layers
    def _add(self, desc, inputs, weight=None, bias=None):
        ins = (ctypes.c_int32 * len(inputs))(*inputs)
        wptr = None
        if weight is not None:
            w = np.ascontiguousarray(weight, dtype=_STORAGE[self.dtype])
            self._keep = w
            wptr = ctypes.c_void_p(w.ctypes.data)
        bptr = None
        if bias is not None:
            b = np.ascontiguousarray(bias, dtype=np.float32)
            self._keepb = b
            bptr = b.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
        out = ctypes.c_int32()
        N.check(self.lib.sn_add_layer(self._g, ctypes.byref(desc), ins, len(inputs), wptr, bptr,
                                      ctypes.byref(out)))
        return out.value

    def add_conv(self, inp, weight, bias, stride=1, pad=0, groups=1, act="none", residual=None):
        """Convolution; ``residual`` (a layer id) is added before the activation."""
        k, _, r, s = weight.shape
        d = N.LayerDesc(N.L_CONV2D, k, r, s, stride, pad, groups, N.ACT[act])
        ins = [inp] if residual is None else [inp, residual]
        return self._add(d, ins, weight, bias)

    def add_projected_conv(self, inp, shortcut, weight, bias, proj_weight, proj_bias, stride=1, pad=0,
                           act="none", proj_stride=1):
        """Convolution of ``inp`` plus a 1x1 projection of ``shortcut`` (at
        ``proj_stride``, no padding), both biases, then the activation."""
        k, _, r, s = weight.shape
        d = N.LayerDesc(N.L_CONV2D, k, r, s, stride, pad, 1, N.ACT[act])
        st = _STORAGE[self.dtype]
        w = np.ascontiguousarray(weight, dtype=st)
        wp = np.ascontiguousarray(np.asarray(proj_weight).reshape(k, -1), dtype=st)
        fp = ctypes.POINTER(ctypes.c_float)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        bp = None if proj_bias is None else np.ascontiguousarray(proj_bias, dtype=np.float32)
        self._keepp = (w, wp, b, bp)
        out = ctypes.c_int32()
        N.check(self.lib.sn_add_projected_conv(
            self._g, ctypes.byref(d), inp, shortcut, proj_stride, ctypes.c_void_p(w.ctypes.data),
            None if b is None else b.ctypes.data_as(fp), ctypes.c_void_p(wp.ctypes.data),
            None if bp is None else bp.ctypes.data_as(fp), ctypes.byref(out)))
        return out.value

    def add_maxpool(self, inp, k=3, stride=2, pad=1):
        return self._add(N.LayerDesc(N.L_MAXPOOL, 0, k, k, stride, pad, 1, 0), [inp])

    def add_gap(self, inp):
        return self._add(N.LayerDesc(N.L_GAP, 0, 0, 0, 1, 0, 1, 0), [inp])

    def add_add(self, a, b, act="none"):
        return self._add(N.LayerDesc(N.L_ADD, 0, 0, 0, 1, 0, 1, N.ACT[act]), [a, b])

    def add_fc(self, inp, weight, bias, act="none"):
        k = weight.shape[0]
        return self._add(N.LayerDesc(N.L_FC, k, 1, 1, 1, 0, 1, N.ACT[act]), [inp], weight, bias)

    def add_input(self, c, h, w):
        """A further net input N x c x h x w (run dtype, NCHW); returns its layer id."""
        out = ctypes.c_int32()
        N.check(self.lib.sn_add_input(self._g, c, h, w, ctypes.byref(out)))
        self.in_shapes.append((self.in_shape[0], c, h, w))
        return out.value

    def mark_output(self, layer):
        """Make ``layer`` the next net output (default: the last layer only)."""
        N.check(self.lib.sn_mark_output(self._g, layer))

    def num_io(self):
        a, b = ctypes.c_int32(), ctypes.c_int32()
        N.check(self.lib.sn_num_io(self._g, ctypes.byref(a), ctypes.byref(b)))
        return a.value, b.value

    def add_spec(self, layer, weight=None, bias=None):
        """Add one layer given as a ``workloads`` spec dict."""
        t = layer["type"]
        if t == "input":
            return self.add_input(*layer["chw"])
        if t == "conv" and layer.get("proj"):
            return self.add_projected_conv(layer["in"][0], layer["in"][1], weight[0], bias[0], weight[1], bias[1],
                                           layer["stride"], layer["pad"], layer["act"], layer["proj"]["stride"])
        if t == "conv":
            res = layer["in"][1] if len(layer["in"]) > 1 else None
            return self.add_conv(layer["in"][0], weight, bias, layer["stride"], layer["pad"],
                                 layer["groups"], layer["act"], res)
        if t == "maxpool":
            return self.add_maxpool(layer["in"][0], layer["k"], layer["stride"], layer["pad"])
        if t == "gap":
            return self.add_gap(layer["in"][0])
        if t == "add":
            return self.add_add(layer["in"][0], layer["in"][1], layer.get("act", "none"))
        if t == "fc":
            return self.add_fc(layer["in"][0], weight, bias, layer.get("act", "none"))
        raise ValueError(t)

    # ---------------------------------------------------------------- tuning
    def profile(self, warmup=5, reps=20, stream=None):
        N.check(self.lib.sn_profile(self._g, warmup, reps, _stream_ptr(stream)))

    def costs(self):
        n = ctypes.c_size_t()
        rc = self.lib.sn_get_costs(self._g, None, 0, ctypes.byref(n))
        if rc not in (0, -6):
            N.check(rc)
        buf = ctypes.create_string_buffer(n.value)
        N.check(self.lib.sn_get_costs(self._g, buf, n.value, ctypes.byref(n)))
        return json.loads(buf.value.decode())

    def set_costs(self, costs):
        s = costs if isinstance(costs, str) else json.dumps(costs)
        N.check(self.lib.sn_set_costs(self._g, s.encode()))

    def select(self, mode="dprs", layout="NCHW", algo="igemm"):
        if mode == "dprs":
            N.check(self.lib.sn_select_path(self._g, N.SELECT_DPRS, 0, 0))
        else:
            lay = N.LAYOUT[layout] if isinstance(layout, str) else layout
            alg = N.ALGO[algo] if isinstance(algo, str) else algo
            N.check(self.lib.sn_select_path(self._g, N.SELECT_FIXED, lay, alg))

    def profile_integrated(self, warmup=3, reps=10, stream=None):
        """Integrated profiling (Sec. III-C): time the candidate paths end to
        end and select the fastest; reps=0 only lists the candidates.
        Returns the candidates as dicts (path, model_ns, measured_ns, kind, a, b)."""
        n = ctypes.c_int32()
        sp = _stream_ptr(stream) if reps > 0 and self.device >= 0 else ctypes.c_void_p(0)
        N.check(self.lib.sn_profile_integrated(self._g, warmup, reps, sp, ctypes.byref(n)))
        nl = self.num_layers()
        out = []
        for i in range(n.value):
            ids = (ctypes.c_int32 * nl)()
            mo, me = ctypes.c_int64(), ctypes.c_int64()
            kab = (ctypes.c_int32 * 3)()
            N.check(self.lib.sn_integrated_candidate(self._g, i, ids, nl, ctypes.byref(mo),
                                                     ctypes.byref(me), kab))
            out.append({"path": list(ids), "model_ns": mo.value, "measured_ns": me.value,
                        "kind": "dprs" if kab[0] == 0 else "fixed", "a": kab[1], "b": kab[2]})
        return out

    def refine_in_path(self, tol_permille=150, max_alts=3, reps=15, stream=None):
        """In-path refinement of the selected path (integrated profiling of
        Sec. III-C applied one layer at a time): near-tied routines of each
        layer's schema are timed inside the whole path and a clear winner
        replaces the selected routine, if the refined path also wins end to
        end.  Returns the number of layers whose routine changed."""
        n = ctypes.c_int32()
        sp = _stream_ptr(stream) if self.device >= 0 else ctypes.c_void_p(0)
        N.check(self.lib.sn_refine_in_path(self._g, int(tol_permille), int(max_alts), int(reps), sp,
                                           ctypes.byref(n)))
        return n.value

    def set_path(self, ids):
        arr = (ctypes.c_int32 * len(ids))(*ids)
        N.check(self.lib.sn_set_path(self._g, arr, len(ids)))

    def path(self):
        n = self.num_layers()
        arr = (ctypes.c_int32 * n)()
        t = ctypes.c_int64()
        N.check(self.lib.sn_get_path(self._g, arr, n, ctypes.byref(t)))
        return list(arr), t.value

    # ---------------------------------------------------------------- queries
    def num_layers(self):
        n = ctypes.c_int32()
        N.check(self.lib.sn_num_layers(self._g, ctypes.byref(n)))
        return n.value

    def routines(self, layer):
        c = ctypes.c_int32()
        N.check(self.lib.sn_num_routines(self._g, layer, ctypes.byref(c)))
        out = []
        for i in range(c.value):
            d = N.RoutineDesc()
            N.check(self.lib.sn_routine_info(self._g, layer, i, ctypes.byref(d)))
            out.append({"id": d.id, "layout": d.layout, "algo": d.algo, "param": d.param,
                        "dtype": d.dtype, "schema": d.schema, "cost_ns": d.cost_ns, "ws_bytes": d.ws_bytes,
                        "name": d.name.decode()})
        return out

    def layer_shape(self, layer):
        arr = (ctypes.c_int32 * 4)()
        N.check(self.lib.sn_layer_shape(self._g, layer, arr))
        return tuple(arr)

    def output_shape(self):
        return self.layer_shape(self.num_layers() - 1)

    def dp_stats(self, layer):
        s, c = ctypes.c_int64(), ctypes.c_int64()
        N.check(self.lib.sn_dp_stats(self._g, layer, ctypes.byref(s), ctypes.byref(c)))
        return s.value, c.value

    # ---------------------------------------------------------------- inference
    def _torch_dtype(self):
        import torch
        return {N.F32: torch.float32, N.F16: torch.float16, N.BF16: torch.bfloat16}[self.dtype]

    def empty_output(self, shape=None):
        import torch
        n, c, h, w = self.output_shape() if shape is None else shape
        shape = (n, c) if h == 1 and w == 1 else (n, c, h, w)
        return torch.empty(shape, dtype=self._torch_dtype(), device=f"cuda:{self.device}")

    def run_mimo(self, xs, outs=None, output_layers=None, stream=None):
        """Inference of a net with several inputs / outputs: ``xs`` are the
        NCHW device tensors of the net inputs in order; returns the outputs
        (``output_layers``: their layer ids, for the shapes)."""
        n_in, n_out = self.num_io()
        assert len(xs) == n_in
        if outs is None:
            assert output_layers is not None and len(output_layers) == n_out
            outs = [self.empty_output(self.layer_shape(l)) for l in output_layers]
        for x, shp in zip(xs, self.in_shapes):
            assert x.is_contiguous() and x.dtype == self._torch_dtype() and tuple(x.shape) == tuple(shp)
        pin = (ctypes.c_void_p * n_in)(*[x.data_ptr() for x in xs])
        pout = (ctypes.c_void_p * n_out)(*[o.data_ptr() for o in outs])
        N.check(self.lib.sn_run_mimo(self._g, pin, n_in, pout, n_out, _stream_ptr(stream)))
        return outs

    def run(self, x, out=None, stream=None):
        """Enqueue inference of NCHW device tensor x; returns the output tensor."""
        if out is None:
            out = self.empty_output()
        assert x.is_contiguous() and out.is_contiguous()
        assert x.dtype == self._torch_dtype() and tuple(x.shape) == tuple(self.in_shape)
        N.check(self.lib.sn_run(self._g, ctypes.c_void_p(x.data_ptr()),
                                ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream)))
        return out

    def run_noalloc(self, x, out, stream=None):
        """sn_run with the intermediate tensors in the library's static
        per-device region (no allocation); ``out`` must be given."""
        assert x.is_contiguous() and out.is_contiguous()
        assert x.dtype == self._torch_dtype() and tuple(x.shape) == tuple(self.in_shape)
        N.check(self.lib.sn_run_noalloc(self._g, ctypes.c_void_p(x.data_ptr()),
                                        ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream)))
        return out

    def plan_launches(self):
        """The layer of each kernel launch of one run, in launch order."""
        n = ctypes.c_int32()
        N.check(self.lib.sn_plan_launches(self._g, None, 0, ctypes.byref(n)))
        arr = (ctypes.c_int32 * max(n.value, 1))()
        N.check(self.lib.sn_plan_launches(self._g, arr, n.value, ctypes.byref(n)))
        return list(arr)[:n.value]

    def layer_output(self, layer, stream=None):
        """The stored bytes of a layer's output after a run (its routine's
        layout; NC8HW8 channels padded), as (uint8 device tensor, layout)."""
        import torch
        nb, lay = ctypes.c_size_t(), ctypes.c_int32()
        N.check(self.lib.sn_layer_output(self._g, layer, None, 0, ctypes.byref(nb), ctypes.byref(lay),
                                         _stream_ptr(stream)))
        buf = torch.empty(max(nb.value, 1), dtype=torch.uint8, device=f"cuda:{self.device}")
        N.check(self.lib.sn_layer_output(self._g, layer, ctypes.c_void_p(buf.data_ptr()), nb.value,
                                         None, None, _stream_ptr(stream)))
        return buf[:nb.value], lay.value

    def run_timed(self, x, out=None, stream=None, reps=1):
        """Synchronous run with every layer's launches repeated ``reps`` times
        back to back; returns (out, per-layer milliseconds per repetition)."""
        if out is None:
            out = self.empty_output()
        n = self.num_layers()
        ms = (ctypes.c_float * n)()
        N.check(self.lib.sn_run_timed(self._g, ctypes.c_void_p(x.data_ptr()),
                                      ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream),
                                      int(reps), ms, n))
        return out, list(ms)


def to_device(arr, dtype, device=0):
    """Copy a host array of stored ``dtype`` values (bf16 as uint16 bits) to a
    torch device tensor of the matching dtype."""
    import torch
    a = np.ascontiguousarray(arr)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(f"cuda:{device}")
    return torch.from_numpy(a).to(f"cuda:{device}")


def build_from_spec(spec, tensors=None, device=0, layouts=None, algos=None, params=True, dtypes=None,
                    ws_limit=None):
    """Create a graph from a ``workloads`` net spec.  ``tensors`` holds the
    generated weights (``workloads.generate``); host-only graphs (device -1)
    may pass None and get zero weights of the right shapes.  ``dtypes``: the
    element types routines may compute in (default: the spec's dtype only);
    a spec's ``outputs`` list marks the net outputs; ``ws_limit``: the
    largest routine workspace admitted (bytes; None = no limit)."""
    from workloads import weight_shapes
    n = spec["batch"]
    c, h, w = spec["in_chw"]
    g = Graph(spec["dtype"], n, c, h, w, device=device,
              layouts=spec.get("layouts") if layouts is None else layouts,
              algos=spec.get("algos") if algos is None else algos, params=params,
              dtypes=spec.get("dtypes") if dtypes is None else dtypes, ws_limit=ws_limit)
    shapes = weight_shapes(spec)
    for i, layer in enumerate(spec["layers"]):
        wt = bt = None
        if shapes[i] is not None:
            if tensors is not None:
                wt, bt = tensors["w"][i], tensors["b"][i]
            else:
                wt = np.zeros(shapes[i][0], dtype=_STORAGE[g.dtype])
                bt = np.zeros(shapes[i][1], dtype=np.float32)
                if len(shapes[i]) == 3:  # a projected shortcut's weights too
                    wt = (wt, np.zeros(shapes[i][2], dtype=_STORAGE[g.dtype]))
                    bt = (bt, np.zeros(shapes[i][1], dtype=np.float32))
        g.add_spec(layer, wt, bt)
    for o in spec.get("outputs", []):
        g.mark_output(o)
    return g
