"""The point-cloud networks of the synthetic workloads, composed from C-ABI
calls only (every arithmetic step runs in libmesorasi.so; torch provides
device memory, streams and events).

Delayed aggregation (Sec. 4.1): the neighbor search N does not depend on
the MLP F, so all searches run on a side stream while F runs on the main
stream; an event joins them right before each aggregation A.  For
PointNet++ the whole xyz chain (FPS -> ball query -> FPS of the next
level ...) depends on coordinates only and runs ahead (Sec. 5.1 "Work
Flow"); for DGCNN each layer's kNN overlaps that layer's MLP.  The
conventional path (Eq. (1)) serialises N -> A -> F per module.  The
limited order (delayed="ltd", Sec. 7.3) hoists only each PointNet++
module's first-layer product onto the input points (overlapping the
search), subtracts the centroid term before bias and ReLU, and runs the
remaining layers on the neighbor rows; for DGCNN's one-layer EdgeConv it
is the delayed order.

All intermediate buffers are allocated once per input shape and kept, so a
forward pass only enqueues kernels and can be captured into a HIP graph
(:meth:`Net.capture`).
"""
from __future__ import annotations

import numpy as np
import torch

from . import ops
from ._lib import F32, BF16


class Net:
    def __init__(self, spec: dict, weights: dict, delayed: bool = True, device="cuda", debug: bool = False,
                 fuse_aggregation: bool = True, fp_coarse_min_rows: int = 4096, fps_prefix: bool = True,
                 fuse_head: bool = True, bq_grid_min_n: int = 4096):
        self.spec = spec
        self.bq_grid_min_n = bq_grid_min_n
        self.fuse_aggregation = fuse_aggregation
        self.fuse_head = fuse_head
        self.fp_coarse_min_rows = fp_coarse_min_rows
        self.fps_prefix = fps_prefix
        self._grid0 = None
        self.delayed = delayed
        self.device = torch.device(device)
        self.dt = BF16 if spec.get("dtype") == "bf16" else F32
        self.side = torch.cuda.Stream(device=self.device)
        self._bufs: dict[str, torch.Tensor] = {}
        self._views: dict[str, torch.Tensor] = {}
        self.debug = debug
        self._range_counts: dict[str, torch.Tensor] = {}
        self._params(weights)

    # -- debug index checks ---------------------------------------------------
    def _check_range(self, name, idx, bound):
        """debug: count entries of a search output outside [0, bound) on the
        stream that produced it (read back by index_errors())."""
        if self.debug:
            self._range_counts[name] = ops.count_out_of_range(idx, bound, out=self._buf(f"rc_{name}", (),
                                                                                         torch.int32))

    def index_errors(self) -> dict:
        """After a debug forward: {output name: entries out of range}, only
        the nonzero ones (synchronises)."""
        torch.cuda.synchronize(self.device)
        return {k: int(v.item()) for k, v in self._range_counts.items() if int(v.item())}

    # -- buffers ------------------------------------------------------------
    def _buf(self, name, shape, dtype=torch.float32):
        t = self._bufs.get(name)
        if t is None or tuple(t.shape) != tuple(shape) or t.dtype != dtype:
            t = torch.empty(shape, dtype=dtype, device=self.device)
            self._bufs[name] = t
        return t

    def _ws(self, name, nbytes):
        t = self._bufs.get(name)
        if t is None or t.numel() < nbytes:
            t = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=self.device)
            self._bufs[name] = t
        return t

    def _params(self, weights):
        raise NotImplementedError

    def forward(self, xyz, feat=None) -> dict:
        raise NotImplementedError

    __call__ = forward

    def capture(self, xyz, feat=None):
        """Warm up, then capture one forward into a CUDA/HIP graph.  Returns
        (graph, outputs); graph.replay() recomputes outputs in place from the
        same input tensors."""
        self.forward(xyz, feat)
        torch.cuda.synchronize(self.device)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            outs = self.forward(xyz, feat)
        return graph, outs


class PointNet2(Net):
    """Set-abstraction stack, optionally followed by a group-all module and
    an FC head (classifier), or by feature propagation and a per-point head
    (segmentation)."""

    def _params(self, w):
        P = lambda Wb: ops.MLPParams(Wb[0], Wb[1], dtype=self.dt, device=self.device)
        self.sa = [P(Wb) for Wb in w["sa"]]
        self.ga = P(w["group_all"]) if "group_all" in w else None
        self.fc = P(w["fc"]) if "fc" in w else None
        self.fp = [P(Wb) for Wb in w.get("fp", [])]
        self.head = P(w["head"]) if "head" in w else None
        # Feature propagation reads [interpolated | skip] rows.  The skip of
        # FP level k is SA level L - 2 - k's output, which that level writes
        # straight into the columns after the interpolation of one buffer,
        # so the MLP reads one contiguous source; the last level's skip is
        # the input features, taken first (with the first layer's weight
        # columns permuted to match) so that the layer's wide source is a
        # plain row-major one.
        L = len(self.spec["sa"])
        self.skip_of = {}
        for k in range(len(self.fp)):
            s = L - 2 - k
            ci = self.sa[L - 1].c_out if k == 0 else self.fp[k - 1].c_out
            if s >= 0:
                self.skip_of[s] = (k, ci)
        self.fp_last_feat_first = None
        if self.fp and self.spec.get("n_feat"):
            Ws, bs = w["fp"][-1]
            W0 = np.asarray(Ws[0], np.float32)
            ci = self.fp[-2].c_out if len(self.fp) > 1 else self.sa[L - 1].c_out
            W0p = np.ascontiguousarray(np.concatenate([W0[:, ci:], W0[:, :ci]], 1))
            self.fp_last_feat_first = P(([W0p] + list(Ws[1:]), bs))
        # Feature propagation's first layer on [interp(f) | s] rows is
        # W1a interp(f) + W1b s + b1 = interp(W1a f) + (W1b s + b1): the
        # interpolation is a convex combination.  So W1a f can be taken on
        # the coarse points (4x fewer rows), W1b s + b1 as soon as the skip
        # features exist (off the critical path), and one kernel forms the
        # layer (mesorasi_interpolate3_add).  fp32 levels of two or more
        # layers with a skip.
        self.fp_split = [None] * len(self.fp)
        if self.dt == F32:
            for k, (Ws, bs) in enumerate(w.get("fp", [])):
                ci = self.sa[L - 1].c_out if k == 0 else self.fp[k - 1].c_out
                W1 = np.asarray(Ws[0], np.float32)
                if len(Ws) < 2 or W1.shape[1] <= ci:
                    continue
                self.fp_split[k] = dict(
                    a=ops.MLPParams([np.ascontiguousarray(W1[:, :ci])], [None], device=self.device),
                    b=ops.MLPParams([np.ascontiguousarray(W1[:, ci:])], [bs[0]], device=self.device),
                    rest=ops.MLPParams(Ws[1:], bs[1:], device=self.device))
                if k == len(self.fp) - 1 and "head" in w:
                    # the level's remaining layers followed by the head, one MLP
                    hW, hb = w["head"]
                    self.fp_split[k]["rest_head"] = ops.MLPParams(list(Ws[1:]) + list(hW), list(bs[1:]) + list(hb),
                                                                  device=self.device)
        if self.delayed == "ltd":
            # limited order (Sec. 7.3): the first layer's product on the input
            # points and on the centroids, its bias, and the remaining layers
            if self.dt != F32:
                raise ValueError("the limited delayed order is built for fp32 networks")
            self.ltd = []
            for Ws, bs in w["sa"]:
                if len(Ws) < 2:
                    raise ValueError("a one-layer module's limited order is its delayed order")
                W1 = np.asarray(Ws[0], np.float32)
                self.ltd.append(dict(
                    first=ops.MLPParams([W1], [None], device=self.device),
                    cen=ops.MLPParams([np.ascontiguousarray(W1[:, :3])], [None], device=self.device),
                    b1=torch.as_tensor(np.asarray(bs[0], np.float32)).to(self.device).contiguous(),
                    rest=ops.MLPParams(Ws[1:], bs[1:], device=self.device)))

    def _search_chain(self, xyz, B):
        """The sampling on the side stream, then (with fps_prefix) the ball
        queries of every level after the first, then the
        feature-propagation 3-NN searches, which need only the sampled
        coordinates.  With fps_prefix every level's centroids are a prefix
        of the first level's, so the whole chain waits only for the first
        sampling; the first level's ball query runs on the main stream right
        after it.  Without it, each level samples the previous level's
        centroids with the sampling kernel and every ball query runs on the
        main stream right before the aggregation that reads it (no sampling
        waits for a ball query).  Each cross-stream wait costs the main
        stream several microseconds in a graph replay, so the main stream
        waits at most once per event; the side stream is joined once more
        at the start of feature propagation.  (Two branches: a graph replay
        maps further branches onto shared hardware queues, which can put a
        main-stream MLP behind an FPS.)"""
        main, side = torch.cuda.current_stream(self.device), self.side
        side.wait_stream(main)
        ev_fps = []
        self._bq_done = set()
        self._waited = set()
        L = len(self.spec["sa"])
        with torch.cuda.stream(side):
            p = xyz
            lv = [xyz]
            for i, m in enumerate(self.spec["sa"]):
                idx = self._buf(f"idx{i}", (B, m["M"]), torch.int32)
                cx = self._buf(f"cxyz{i}", (B, m["M"], 3))
                if i == 0 or not self.fps_prefix:
                    ws = self._ws(f"ws_fps{i}", ops.fps_workspace_bytes(B, p.shape[1], m["M"]))
                    ops.fps(p, m["M"], out_idx=idx, out_xyz=cx, ws=ws)
                    self._check_range(f"idx{i}", idx, p.shape[1])
                    e = torch.cuda.Event()
                    e.record(side)
                    ev_fps.append(e)
                p = cx
                lv.append(cx)
            if self.fps_prefix and L > 1:
                # level i samples level i-1's centroids, themselves a
                # sampling in selection order: its first M, exactly -- all
                # levels after the first from the first one, in one launch
                sa = self.spec["sa"]
                ops.fps_prefix_levels(self._bufs["idx0"], self._bufs["cxyz0"], [m["M"] for m in sa[1:]],
                                      out_idx=[self._bufs[f"idx{i}"] for i in range(1, L)],
                                      out_xyz=[self._bufs[f"cxyz{i}"] for i in range(1, L)])
                for i in range(1, L):
                    self._check_range(f"idx{i}", self._bufs[f"idx{i}"], sa[i - 1]["M"])
            if self.fps_prefix and L > 1:
                for i in range(1, L):
                    self._issue_ball_query(i, lv[i])
                    self._bq_done.add(i)
                e = torch.cuda.Event()
                e.record(side)
                ev_fps += [e] * (L - 1)
            if self.fp:
                n = len(self.fp)
                for i in range(n):
                    fine, coarse = lv[len(lv) - 2 - i], lv[len(lv) - 1 - i]
                    nn = self._buf(f"nn{i}", (B, fine.shape[1], 3), torch.int32)
                    nd = self._buf(f"nnd{i}", (B, fine.shape[1], 3))
                    ops.three_nn(fine, coarse, out_nit=nn, out_dist=nd)
                    self._check_range(f"nn{i}", nn, coarse.shape[1])
        self._ev_fps = ev_fps
        return ev_fps

    def _issue_ball_query(self, i, p):
        """Level i's ball query on the current stream (against the input
        cloud's prebuilt grid for the first level when there is one)."""
        m = self.spec["sa"][i]
        B, N = p.shape[0], p.shape[1]
        nit = self._buf(f"nit{i}", (B, m["M"], m["K"]), torch.int32)
        if i == 0 and self._grid0 is not None:
            ops.ball_query_grid(p, self._bufs["cxyz0"], m["radius"], m["K"], self._grid0, out=nit)
        else:
            ws = self._ws(f"ws_bq{i}", ops.ball_query_workspace_bytes(B, N, m["M"]))
            ops.ball_query(p, self._bufs[f"cxyz{i}"], m["radius"], m["K"], out=nit, ws=ws)
        self._check_range(f"nit{i}", nit, N)

    def _ball_query(self, i, p):
        """Level i's ball query: on the main stream after level i's sampling
        (issued once per forward, at its first reader), or, when the search
        chain already issued it, the wait for it."""
        if i in self._bq_done:
            self._wait_fps(i)
            return
        self._bq_done.add(i)
        self._wait_fps(i)
        self._issue_ball_query(i, p)

    def _wait_fps(self, i):
        """The main stream waits for level i's sampling, once per event per
        forward (a repeated wait would add a cross-stream edge to the graph)."""
        e = self._ev_fps[i]
        if id(e) not in self._waited:
            self._waited.add(id(e))
            torch.cuda.current_stream(self.device).wait_event(e)

    def _fp_coarse(self, k, rows):
        """FP level k takes its first product on the coarse points."""
        return self.fp_split[k] is not None and rows >= self.fp_coarse_min_rows

    def _fp_pre(self, s, skip):
        """W1b s + b1 of the FP level whose skip is SA level s's output (s =
        -1: the input features), issued as soon as that output exists: on
        the main stream for the input features (idle while the first
        sampling runs), on the side stream for an SA level's output (off
        the main stream's path; joined at the start of feature
        propagation)."""
        if not self.fp or skip is None:
            return
        k = len(self.spec["sa"]) - 2 - s
        if not 0 <= k < len(self.fp):      # the last SA level's output is no skip
            return
        B, Nf = skip.shape[0], skip.shape[1]
        if not self._fp_coarse(k, B * Nf):
            return
        sp = self.fp_split[k]
        pre = self._buf(f"fpp{k}", (B, Nf, sp["b"].c_out))
        ws = self._ws(f"ws_fpp{k}", ops.mlp_workspace_bytes(B * Nf, sp["b"]))
        if s < 0:
            ops.pointwise_mlp(skip, sp["b"], relu_mask=0, out=pre, ws=ws)
            return
        main, side = torch.cuda.current_stream(self.device), self.side
        e = torch.cuda.Event()
        e.record(main)
        with torch.cuda.stream(side):
            side.wait_event(e)
            ops.pointwise_mlp(skip, sp["b"], relu_mask=0, out=pre, ws=ws)

    def _fused_into(self, i):
        """Level i's MLP takes level i - 1's aggregation in its loader."""
        return (self.fuse_aggregation and self.dt == F32 and self.delayed is True
                and ops.aggregate_mlp_supported(self.sa[i], self.sa[i - 1].c_out))

    def _sa_levels(self, xyz, feat):
        B = xyz.shape[0]
        main = torch.cuda.current_stream(self.device)
        ev_fps = self._search_chain(xyz, B)
        # the input cloud binned for the first ball query (main stream, while
        # the first sampling runs on the side stream)
        self._grid0 = None
        if self.spec["sa"] and xyz.shape[1] >= self.bq_grid_min_n:
            N = xyz.shape[1]
            ws = self._ws("ws_grid0", ops.ball_query_grid_workspace_bytes(B, N))
            self._grid0 = ops.ball_query_grid_build(xyz, self.spec["sa"][0]["radius"], ws=ws)
        self._fp_pre(-1, feat)
        levels = [(xyz, feat)]
        p, f = xyz, feat
        for i, m in enumerate(self.spec["sa"]):
            prm = self.sa[i]
            N = p.shape[1]
            # p = the previous level's centroids: already ordered, since the
            # previous level's ball query (main stream) waited for its FPS (a
            # redundant wait would add a cross-stream edge to the graph)
            idx, cx = self._bufs[f"idx{i}"], self._bufs[f"cxyz{i}"]
            nit = self._buf(f"nit{i}", (B, m["M"], m["K"]), torch.int32)
            if i in self.skip_of:
                k, ci = self.skip_of[i]
                cat = self._buf(f"cat{k}", (B, m["M"], ci + prm.c_out))
                out = cat[..., ci:]
            else:
                out = self._buf(f"f{i}", (B, m["M"], prm.c_out))
            self._views[f"f{i}"] = out
            if self.delayed == "ltd":
                L = self.ltd[i]
                c1 = L["first"].c_out
                p1 = self._buf(f"p1_{i}", (B, N, c1))
                ws = self._ws(f"ws_p1_{i}", ops.mlp_workspace_bytes(B * N, L["first"]))
                ops.pointwise_mlp(p, L["first"], x1=f, relu_mask=0, out=p1, ws=ws)   # overlaps the search chain
                q = self._buf(f"q_{i}", (B, m["M"], c1))
                self._wait_fps(i)
                ws = self._ws(f"ws_q_{i}", ops.mlp_workspace_bytes(B * m["M"], L["cen"]))
                ops.pointwise_mlp(cx, L["cen"], relu_mask=0, out=q, ws=ws)
                self._ball_query(i, p)
                ws = self._ws(f"ws_sa{i}", ops.ltd_workspace_bytes(B, m["M"], m["K"], L["rest"]))
                ops.ltd_module(p1, q, nit, L["rest"], b1=L["b1"], out=out, ws=ws)
                self._fp_pre(i, out)
            elif self.delayed:
                # F on all N input points -> PFT, overlapping the search chain
                pft_dt = torch.bfloat16 if self.dt == BF16 else torch.float32
                pft = self._buf(f"pft{i}", (B, N, prm.c_out), pft_dt)
                if i > 0 and self._fused_into(i):
                    # the previous level's aggregation happens in this MLP's
                    # loader (Sec. 5.2), which also stores it (f, the level's
                    # output, is the next point set's features and a skip)
                    self._ball_query(i - 1, levels[i - 1][0])
                    ops.aggregate_mlp(p, self._bufs[f"pft{i - 1}"], self._bufs[f"nit{i - 1}"],
                                      self._bufs[f"idx{i - 1}"], prm, out=pft, agg_out=f)
                    self._fp_pre(i - 1, f)
                else:
                    ws = self._ws(f"ws_sa{i}", ops.mlp_workspace_bytes(B * N, prm))
                    ops.pointwise_mlp(p, prm, x1=f, out_dtype=self.dt, out=pft, ws=ws)
                if not (i + 1 < len(self.spec["sa"]) and self._fused_into(i + 1)):
                    self._ball_query(i, p)
                    ops.aggregate_max(pft, nit, cidx=idx, sign=-1, out=out)
                    self._fp_pre(i, out)
            else:
                self._ball_query(i, p)
                ws = self._ws(f"ws_sa{i}", ops.conventional_workspace_bytes(B, m["M"], m["K"], prm))
                ops.conventional_module(nit, prm, xyz=p, feat=f, cxyz=cx, grouping=0, out=out, ws=ws)
                self._fp_pre(i, out)
            p, f = cx, out
            levels.append((p, f))
        return levels

    def forward(self, xyz, feat=None) -> dict:
        B = xyz.shape[0]
        levels = self._sa_levels(xyz, feat)
        res = {}
        for i in range(len(self.spec["sa"])):
            for k in ("idx", "nit", "cxyz"):
                res[f"{k}{i}"] = self._bufs[f"{k}{i}"]
            res[f"f{i}"] = self._views[f"f{i}"]
        p, f = levels[-1]
        res["out"] = f
        if self.ga is not None:
            g = self._buf("global", (B, self.ga.c_out))
            ws = self._ws("ws_ga", ops.mlp_workspace_bytes(B * p.shape[1], self.ga, p.shape[1]))
            ops.pointwise_mlp(p, self.ga, x1=f, pool_group=p.shape[1], out=g, ws=ws)
            res["global"] = res["out"] = g
            if self.fc is not None:
                logits = self._buf("logits", (B, self.fc.c_out))
                ws = self._ws("ws_fc", ops.mlp_workspace_bytes(B, self.fc))
                ops.pointwise_mlp(g, self.fc, relu_mask=(1 << (self.fc.n - 1)) - 1, out=logits, ws=ws)
                res["out"] = logits
        if self.fp:
            main = torch.cuda.current_stream(self.device)
            # the side stream's searches and skip products, all done long
            # before: one join
            e = torch.cuda.Event()
            e.record(self.side)
            main.wait_event(e)
            coarse_xyz, coarse_f = levels[-1]
            L = len(self.spec["sa"])
            for i, prm in enumerate(self.fp):
                fine_xyz, fine_f = levels[len(levels) - 2 - i]
                Nf = fine_xyz.shape[1]
                ci = coarse_f.shape[-1]
                s = L - 2 - i
                y = self._buf(f"fp{i}", (B, Nf, prm.c_out))
                if self._fp_coarse(i, B * Nf) and (s >= 0 or fine_f is not None):
                    # first product on the coarse points, then the layer as
                    # interp + (W1b s + b1), ReLU (in place), then the rest
                    sp = self.fp_split[i]
                    g = self._buf(f"fpg{i}", (B, coarse_f.shape[1], sp["a"].c_out))
                    ws = self._ws(f"ws_fpg{i}", ops.mlp_workspace_bytes(B * coarse_f.shape[1], sp["a"]))
                    ops.pointwise_mlp(coarse_f, sp["a"], relu_mask=0, out=g, ws=ws)
                    h = self._bufs[f"fpp{i}"]
                    rh = sp.get("rest_head") if self.fuse_head and self.head is not None else None
                    if B * Nf > 32768 and rh is not None and ops.interpolate3_mlp_supported(rh, B * Nf):
                        # the layer formed in the register MLP's row loader,
                        # then the remaining layers and the head: the logits
                        logits = self._buf("logits", (B, Nf, self.head.c_out))
                        ops.interpolate3_mlp(self._bufs[f"nn{i}"], self._bufs[f"nnd{i}"], g, h, rh,
                                             relu_mask=(1 << (rh.n - 1)) - 1, out=logits)
                        res["out"] = logits
                        return res
                    if B * Nf > 32768 and ops.interpolate3_mlp_supported(sp["rest"], B * Nf):
                        # the layer formed in the register MLP's row loader
                        ops.interpolate3_mlp(self._bufs[f"nn{i}"], self._bufs[f"nnd{i}"], g, h, sp["rest"], out=y)
                    else:
                        ops.interpolate3_add(self._bufs[f"nn{i}"], self._bufs[f"nnd{i}"], g, h, relu=True, out=h)
                        ws = self._ws(f"ws_fp{i}", ops.mlp_workspace_bytes(B * Nf, sp["rest"]))
                        ops.pointwise_mlp(h, sp["rest"], out=y, ws=ws)
                    res[f"fp{i}"] = y
                    coarse_xyz, coarse_f = fine_xyz, y
                    continue
                if s >= 0:   # [interp | skip] in one buffer, the skip already in place
                    cat = self._bufs[f"cat{i}"]
                    interp, x0, x1, p_mlp = cat[..., :ci], cat, None, prm
                elif fine_f is not None and self.fp_last_feat_first is not None:
                    interp = self._buf(f"interp{i}", (B, Nf, ci))
                    x0, x1, p_mlp = fine_f, interp, self.fp_last_feat_first
                else:
                    interp = self._buf(f"interp{i}", (B, Nf, ci))
                    x0, x1, p_mlp = interp, fine_f, prm
                ops.interpolate3_apply(self._bufs[f"nn{i}"], self._bufs[f"nnd{i}"], coarse_f, out=interp)
                ws = self._ws(f"ws_fp{i}", ops.mlp_workspace_bytes(B * Nf, p_mlp))
                ops.pointwise_mlp(x0, p_mlp, x1=x1, out=y, ws=ws)
                res[f"fp{i}"] = y
                coarse_xyz, coarse_f = fine_xyz, y
            logits = self._buf("logits", (B, coarse_f.shape[1], self.head.c_out))
            ws = self._ws("ws_head", ops.mlp_workspace_bytes(B * coarse_f.shape[1], self.head))
            ops.pointwise_mlp(coarse_f, self.head, relu_mask=(1 << (self.head.n - 1)) - 1, out=logits, ws=ws)
            res["out"] = logits
        return res


class DGCNN(Net):
    """EdgeConv stack (kNN in the current feature space), concatenation,
    1x1 convolution to 1024 channels and a global max."""

    def _params(self, w):
        self.k = self.spec["k"]
        self.widths = list(self.spec["edge"])
        self.edge = []
        self.folded = []
        for W, b in w["edge"]:
            Wd = torch.as_tensor(W, dtype=torch.float32).to(self.device).contiguous()
            bd = torch.as_tensor(b, dtype=torch.float32).to(self.device).contiguous()
            self.edge.append(ops.MLPParams([W], [b], dtype=self.dt, device=self.device))
            Wf, bf = ops.edgeconv_fold(Wd, bd)           # [W1 - W2 ; W2], [b ; 0]
            self.folded.append(ops.MLPParams([Wf], [bf], dtype=self.dt, device=self.device))
        self.conv = ops.MLPParams([w["conv"][0]], [w["conv"][1]], dtype=self.dt, device=self.device)

    def forward(self, xyz, feat=None) -> dict:
        B, N, _ = xyz.shape
        main, side = torch.cuda.current_stream(self.device), self.side
        cat = self._buf("cat", (B, N, sum(self.widths)))
        res = {}
        X = xyz
        off = 0
        for l, cout in enumerate(self.widths):
            nit = self._buf(f"nit{l}", (B, N, self.k), torch.int32)
            side.wait_stream(main)                       # X of this layer is ready
            with torch.cuda.stream(side):
                ops.knn(X, X, self.k, out=nit)
                self._check_range(f"nit{l}", nit, N)
                ev = torch.cuda.Event()
                ev.record(side)
            dst = cat[..., off:off + cout]
            if self.delayed:
                P = self._buf(f"P{l}", (B, N, 2 * cout))
                ops.pointwise_mlp(X, self.folded[l], relu_mask=0, out=P)   # [A | Bm] for every point
                main.wait_event(ev)
                ops.aggregate_max(P[..., cout:], nit, cfeat=P[..., :cout], sign=+1, relu=True, out=dst)
            else:
                main.wait_event(ev)
                ws = self._ws(f"ws_e{l}", ops.conventional_workspace_bytes(B, N, self.k, self.edge[l]))
                ops.conventional_module(nit, self.edge[l], feat=X, grouping=1, out=dst, ws=ws)
            res[f"nit{l}"] = nit
            res[f"x{l}"] = dst
            X = dst
            off += cout
        g = self._buf("global", (B, self.conv.c_out))
        ops.pointwise_mlp(cat, self.conv, pool_group=N, out=g)
        res["cat"] = cat
        res["out"] = g
        return res


def build(spec: dict, weights: dict, delayed: bool | str = True, device="cuda", debug: bool = False,
          fuse_aggregation: bool = True, fp_coarse_min_rows: int = 4096, fps_prefix: bool = True,
          fuse_head: bool = True, bq_grid_min_n: int = 4096) -> Net:
    """delayed: True (delayed aggregation), False (conventional) or "ltd"
    (limited delayed aggregation).  debug: every search output is checked
    to lie in range before anything reads through it (index_errors()).
    fuse_aggregation: where the next level's MLP allows it, a level's
    aggregation runs inside that MLP's loader (mesorasi_aggregate_mlp).
    fp_coarse_min_rows: feature-propagation levels of at least this many
    fine rows take their first product on the coarse points
    (mesorasi_interpolate3_add).  fps_prefix: the sampling of every level
    after the first, which samples the previous level's centroids, is taken
    as their first M (mesorasi_fps_prefix, the same result).  fuse_head: the
    last feature-propagation level's remaining layers and the per-point head
    run in one kernel (mesorasi_interpolate3_mlp), so that level's output
    (``fp{n-1}``) is not materialised.  bq_grid_min_n: input clouds of at
    least this many points are binned for the first ball query while the
    first sampling runs (mesorasi_ball_query_grid_build), so that query
    only looks up the cells."""
    args = (spec, weights, delayed, device, debug, fuse_aggregation, fp_coarse_min_rows, fps_prefix, fuse_head,
            bq_grid_min_n)
    if spec["kind"] in ("pointnet2_cls", "pointnet2_seg"):
        return PointNet2(*args)
    if spec["kind"] == "dgcnn":
        return DGCNN(*args)
    raise ValueError(spec["kind"])
