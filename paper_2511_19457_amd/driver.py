"""Per-layer driver: measure -> route -> execute over a layer stack.

For every conv/FC layer (SparOA Section 3.1 features, Section 2.2 quadrants,
Section 5 online execution on one device):
  1. intensity from the shape (host, Eq. 2);
  2. the kernel family the intensity selects (bandwidth when light or
     depthwise, MFMA otherwise) fixes the skip granularity of its zero-skip
     kernel; the input activation is measured at that granularity on the GPU
     (Eq. 1) and the four counts are read back -- the one host/device
     synchronisation per layer;
  3. sparoa_route picks one of the four paths;
  4. the routed kernel runs with the fused epilogue (bias, residual,
     activation), producing the next layer's input.
Max pooling is glue and is not routed.  All computation is in libsparoa.so;
this module only allocates buffers (PyTorch) and sequences the C calls.

With ``routed=True`` steps 2-4 run without the host round trip: the counts
stay in device memory and the routed kernels take the skip decision
themselves (same arithmetic as sparoa_route); a conv/FC whose output feeds a
conv/FC measures that output in its own epilogue (sparoa_*_routed_measured),
so those consumers skip their measurement pass; counts and paths are read
back once, after the whole stack.
"""
import time
from dataclasses import dataclass

import torch

from . import abi
from .stacks import Layer, input_shape, output_shape


@dataclass
class LayerRecord:
    name: str
    kind: str
    rho_e: float = 0.0
    rho_b: float = 0.0
    intensity: float = 0.0
    macs: int = 0
    bytes: int = 0
    path: int = -1
    us: float = 0.0


class Engine:
    """Holds weights and per-layer buffers of one stack on one device."""

    def __init__(self, layers, dtype, device, seed=0, sparsity_thr=0.5, intensity_thr=315.0,
                 mode=abi.ROUTE_BLOCK, weights=None):
        import synth
        self.layers = layers
        self.dtype = dtype
        self.dev = torch.device(device)
        self.s_thr, self.c_thr, self.mode = sparsity_thr, intensity_thr, mode
        self.st = []
        self.acts = [None] * (len(layers) + 1)
        for i, L in enumerate(layers):
            st = {}
            if L.kind != "maxpool":
                s = L.shape
                if L.kind == "conv":
                    d = abi.conv_desc(s["n"], s["cin"], s["h"], s["w"], s["cout"], s["kh"],
                                      s["kw"], s["sh"], s["sw"], s["ph"], s["pw"], 1, 1,
                                      s["groups"], dtype)
                    st["inten"] = abi.sparoa_op_intensity_conv(d)
                    wshape = (s["cout"], s["kh"], s["kw"], s["cin"] // s["groups"])
                    fan_in = s["kh"] * s["kw"] * s["cin"] // s["groups"]
                    st["rows"], st["cols"] = s["n"] * s["h"] * s["w"], s["cin"]
                    fam = abi.PATH_DENSE_BW if (L.depthwise or st["inten"]["intensity"] <
                                                self.c_thr) else abi.PATH_DENSE_MFMA
                    st["br"], st["bc"] = abi.sparoa_conv2d_skip_block(d, fam | 1)
                    ws = max(abi.sparoa_conv2d_workspace_size(d, p) for p in range(4))
                else:
                    d = abi.fc_desc(s["m"], s["k"], s["n"], dtype)
                    st["inten"] = abi.sparoa_op_intensity_fc(d)
                    wshape = (s["n"], s["k"])
                    fan_in = s["k"]
                    st["rows"], st["cols"] = s["m"], s["k"]
                    fam = abi.PATH_DENSE_BW if st["inten"]["intensity"] < self.c_thr \
                        else abi.PATH_DENSE_MFMA
                    st["br"], st["bc"] = abi.sparoa_fc_skip_block(d, fam | 1)
                    ws = max(abi.sparoa_fc_workspace_size(d, p) for p in (fam, fam | 1))
                st["desc"], st["family"] = d, fam
                if weights is not None:
                    w = weights[i].to(self.dev)
                else:
                    w = synth.he_normal(wshape, fan_in, dtype, seed + 1000 + i).to(self.dev)
                st["w"] = w
                if L.kind == "fc" and abi.sparoa_fc_uses_packed(d, fam):
                    wp = torch.empty(abi.sparoa_fc_packed_bytes(d) // w.element_size(),
                                     dtype=dtype, device=self.dev)
                    abi.sparoa_fc_pack_weights(d, w, wp)
                    st["wp"] = wp
                st["counts"] = torch.zeros(4, dtype=torch.int64, device=self.dev)
                st["mask"] = torch.zeros(
                    abi.sparoa_mask_words(st["rows"], st["cols"], st["br"], st["bc"]),
                    dtype=torch.int32, device=self.dev)
                st["ws_bytes"] = ws
                st["path"] = torch.zeros(1, dtype=torch.int32, device=self.dev)
            self.acts[i + 1] = torch.empty(output_shape(L), dtype=dtype, device=self.dev)
            self.st.append(st)
        # one split-K workspace serves every layer (they run in stream order;
        # its contents on entry do not matter)
        self.ws = torch.empty(max([16] + [st.get("ws_bytes", 0) for st in self.st]),
                              dtype=torch.uint8, device=self.dev)
        for st in self.st:
            if "ws_bytes" in st:
                st["ws"] = self.ws
        # Activations a conv/FC produces and some consumer measures at block
        # (1, 8): in routed mode the producer measures them in its epilogue
        # (sparoa_*_routed_measured) and those consumers skip their own pass.
        # Their counters live in one tensor, reset from a template before
        # each routed pass (one kernel for the whole network).
        self.tmeas = {}
        meas = []
        for i, L in enumerate(layers):
            if L.kind == "maxpool":
                continue
            t = i + 1
            if any(layers[k].src == t and layers[k].kind != "maxpool" and
                   (self.st[k]["br"], self.st[k]["bc"]) == (1, 8) for k in range(len(layers))):
                shp = output_shape(L)
                rows = 1
                for v in shp[:-1]:
                    rows *= v
                nb = rows * -(-shp[-1] // 8)
                meas.append((t, [0, rows * shp[-1], nb, nb], abi.sparoa_mask_words(rows, shp[-1], 1, 8)))
        # Every counter of a routed pass -- each layer's own input measurement
        # (rows 0 .. L-1) and the fused output measurements -- starts from its
        # preset {0, numel, nb, nb}: one reset kernel per pass, and the
        # measurement passes need no init launch of their own.
        tmpl = []
        for i, L in enumerate(layers):
            st = self.st[i]
            if L.kind == "maxpool":
                tmpl.append([0, 0, 0, 0])
                continue
            nb = -(-st["rows"] // st["br"]) * -(-st["cols"] // st["bc"])
            tmpl.append([0, st["rows"] * st["cols"], nb, nb])
        tmpl += [m[1] for m in meas]
        # one 128-byte line per counter: a kernel's atomics into its output
        # counters never share a line with the input counters other
        # work-groups of the same kernel read
        pad = [row + [0] * 12 for row in tmpl]
        # then the zeroed count-commit words of every fused output
        # measurement (16 lines each), reset with the counters
        cw_rows = abi.COMMIT_WORDS_BYTES // 128
        pad += [[0] * 16] * (cw_rows * (len(meas) + 1))
        self.ctr_template = torch.tensor(pad, dtype=torch.int64, device=self.dev)
        self.ctr = torch.zeros_like(self.ctr_template)
        for i, L in enumerate(layers):
            if L.kind != "maxpool":
                self.st[i]["counts"] = self.ctr[i, :4]
        cw0 = len(layers) + len(meas)
        # commit words of the standalone input measurements (one call at a
        # time, each leaves them zero): after the fused outputs' words
        self.commit_in = self.ctr[cw0 + cw_rows * len(meas):cw0 + cw_rows * (len(meas) + 1)]
        for j, (t, _, words) in enumerate(meas):
            # the bitmap only where a consumer's skip kernel reads it (FC
            # consumers, implicit-GEMM convs); the others route on the counts
            # and the producer measures counts only
            need_mask = any(layers[k].src == t and layers[k].kind != "maxpool" and
                            self._reads_mask(k) for k in range(len(layers)))
            mask = torch.zeros(words, dtype=torch.int32, device=self.dev) if need_mask else None
            self.tmeas[t] = dict(counts=self.ctr[len(layers) + j, :4], mask=mask,
                                 commit=self.ctr[cw0 + cw_rows * j:cw0 + cw_rows * (j + 1)])
        torch.cuda.synchronize(self.dev)

    def _reads_mask(self, k):
        """Whether layer k's routed call needs its input's bitmap."""
        if self.layers[k].kind != "conv":
            return True
        return abi.sparoa_conv2d_routed_reads_mask(self.st[k]["desc"], self.s_thr, self.c_thr,
                                                   self.mode)

    def reset_counters(self):
        """Preset values of every counter of a routed pass (a kernel, not a
        memset or copy node, so a captured graph replays it safely)."""
        torch.mul(self.ctr_template, 1, out=self.ctr)
        self._measured = {}   # (source tensor, block shape) -> its measurement this pass

    def weights_cpu(self):
        return [st.get("w").cpu() if "w" in st else None for st in self.st]

    def run_layer(self, i, force_path=None):
        """Runs layer i on the activations already in place; returns its record."""
        L, st = self.layers[i], self.st[i]
        x = self.acts[L.src]
        y = self.acts[i + 1]
        rec = LayerRecord(L.name, L.kind)
        if L.kind == "maxpool":
            s = L.shape
            abi.sparoa_maxpool2d(x, s["n"], s["c"], s["h"], s["w"], s["k"], s["s"], s["p"], y)
            return rec
        c = abi.sparoa_measure_sparsity_sync(x, st["rows"], st["cols"], st["br"], st["bc"], 0,
                                             st["counts"], st["mask"])
        inten = st["inten"]
        path = abi.sparoa_route(c, inten, int(L.depthwise), self.s_thr, self.c_thr, self.mode)
        if force_path is not None:
            path = force_path
        res = self.acts[L.res] if L.res is not None else None
        mask = st["mask"] if path & 1 else None
        if L.kind == "conv":
            abi.sparoa_conv2d(st["desc"], path, x, st["w"], None, res, L.act, mask, y, st["ws"])
        else:
            w = st["wp"] if "wp" in st and (path & 2) else st["w"]
            abi.sparoa_fc(st["desc"], path, x, w, None, res, L.act, mask, y, st["ws"])
        rec.rho_e = c["zeros"] / c["numel"]
        rec.rho_b = c["zero_blocks"] / c["num_blocks"] if c["num_blocks"] else 0.0
        rec.intensity, rec.macs, rec.bytes = inten["intensity"], inten["macs"], inten["bytes"]
        rec.path = path
        rec.counts = c
        return rec

    def run_layer_routed(self, i):
        """Runs layer i with device-side routing (no host synchronisation).
        Its input counts and bitmap come from the producer's fused
        measurement when there is one at this layer's block shape, else from
        a measurement pass; its own output is measured in its epilogue when a
        consumer needs it."""
        L, st = self.layers[i], self.st[i]
        x = self.acts[L.src]
        y = self.acts[i + 1]
        if L.kind == "maxpool":
            s = L.shape
            abi.sparoa_maxpool2d(x, s["n"], s["c"], s["h"], s["w"], s["k"], s["s"], s["p"], y)
            return
        src = self.tmeas.get(L.src) if (st["br"], st["bc"]) == (1, 8) else None
        key = (L.src, st["br"], st["bc"])
        if src is not None:
            counts, mask = src["counts"], src["mask"]
        elif key in self._measured and self._measured[key][0] is not st["counts"]:
            counts, mask = self._measured[key]   # another consumer of x measured it this pass
        else:
            counts, mask = st["counts"], st["mask"]
            abi.sparoa_measure_sparsity_preset(x, st["rows"], st["cols"], st["br"], st["bc"],
                                               counts, mask, commit=self.commit_in)
            self._measured[key] = (counts, mask)
        st["used"] = (counts, mask)
        res = self.acts[L.res] if L.res is not None else None
        out = self.tmeas.get(i + 1)
        if L.kind == "conv":
            if out is not None:
                abi.sparoa_conv2d_routed_measured(st["desc"], self.s_thr, self.c_thr, self.mode,
                                                  counts, x, st["w"], None, res, L.act, mask, y,
                                                  out["counts"], out["mask"], st["ws"], st["path"],
                                                  out["commit"])
            else:
                abi.sparoa_conv2d_routed(st["desc"], self.s_thr, self.c_thr, self.mode, counts, x,
                                         st["w"], None, res, L.act, mask, y, st["ws"], st["path"])
        elif out is not None:
            abi.sparoa_fc_routed_measured(st["desc"], self.s_thr, self.c_thr, self.mode, counts, x,
                                          st["w"], st.get("wp"), None, res, L.act, mask, y,
                                          out["counts"], out["mask"], st["ws"], st["path"],
                                          out["commit"])
        else:
            abi.sparoa_fc_routed(st["desc"], self.s_thr, self.c_thr, self.mode, counts, x,
                                 st["w"], st.get("wp"), None, res, L.act, mask, y, st["ws"],
                                 st["path"])

    def forward_routed(self, x):
        """The whole stack with device-side routing and no host synchronisation
        (stream-ordered; safe to capture in a HIP graph).  Returns the output
        activation tensor."""
        self.acts[0] = x
        self.reset_counters()
        for i in range(len(self.layers)):
            self.run_layer_routed(i)
        return self.acts[len(self.layers)]

    def records_from_device(self):
        """Counts and paths of the last routed run, read back after the fact."""
        recs = []
        for L, st in zip(self.layers, self.st):
            rec = LayerRecord(L.name, L.kind)
            if L.kind != "maxpool":
                c = dict(zip(("zeros", "numel", "zero_blocks", "num_blocks"),
                             st.get("used", (st["counts"],))[0].cpu().tolist()))
                rec.counts = c
                rec.rho_e = c["zeros"] / c["numel"]
                rec.rho_b = c["zero_blocks"] / c["num_blocks"] if c["num_blocks"] else 0.0
                inten = st["inten"]
                rec.intensity, rec.macs, rec.bytes = (inten["intensity"], inten["macs"],
                                                      inten["bytes"])
                rec.path = int(st["path"].item())
            recs.append(rec)
        return recs

    def run(self, x, timed=False, routed=False):
        """Full stack on input x (device tensor of the input shape); returns
        (output, records, wall seconds)."""
        assert tuple(x.shape) == input_shape(self.layers) and x.dtype == self.dtype
        self.acts[0] = x
        recs = []
        evs = []
        torch.cuda.synchronize(self.dev)
        t0 = time.perf_counter()
        if routed:
            self.reset_counters()
        for i in range(len(self.layers)):
            if timed:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
            if routed:
                self.run_layer_routed(i)
            else:
                recs.append(self.run_layer(i))
            if timed:
                e1.record()
                evs.append((e0, e1))
        torch.cuda.synchronize(self.dev)
        wall = time.perf_counter() - t0
        if routed:
            recs = self.records_from_device()
        for r, ev in zip(recs, evs):
            r._ev = ev
        if timed:
            for r in recs:
                r.us = r._ev[0].elapsed_time(r._ev[1]) * 1e3
                del r._ev
        return self.acts[len(self.layers)], recs, wall
