"""One GPU's share of one MoE layer, run through the five C-ABI calls.

`LayerShare` owns the device buffers of one share (allocated once with
torch) and enqueues, on the current stream:
    moe_route_topk -> moe_expert_histogram -> moe_permute
    -> moe_grouped_ffn (routed experts) -> moe_combine
with no host synchronisation in between (decode-sized batches stream every
expert group and skip the tiled GEMM launches; at most 64 tokens with k <= 2 the
last two calls are one, moe_grouped_ffn_combine).  The shared experts (always
on, independent of the routing) run one of two ways.  Up to SHARED_IN_FFN_MAX_T
tokens they are leading groups of the routed experts' FFN call
(moe_grouped_ffn_rows_shared: each shared expert cut into blocks of the routed
width f, every token once per block), so the tiles of both fill the GPU
together, and moe_combine_shared adds their slices.  Over longer batches, where
each call fills the GPU by itself, they are a moe_grouped_ffn call of their own
on a second stream forked from the current one after the packaging step and
joined back before the combine, overlapping the routed experts' FFN (whose
launches leave CUs idle) without holding CUs the routing launches wait for;
the fork and join are stream events, so a graph capture of `run` holds both
branches.  The expert placement can be swapped between batches
(`set_placement`) by re-pointing the weight table; nothing is reallocated.
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np
import torch

from . import moe


# Longest batch whose shared experts join the routed experts' FFN call (one call
# for both) rather than run as a call of their own on a second stream.  Measured
# per step, graph replays over rotated weights: Qwen1.5-MoE-shaped batch (T =
# 2048, one shared expert of 4 f) 324 -> 283 us, DeepSeek-V2-Lite-shaped decode
# (T = 256, two shared experts of f) 127 -> 115 us, but its prefill batch (T =
# 8192) 619 -> 628 us: there each call fills the GPU alone and the two streams
# overlap well.
SHARED_IN_FFN_MAX_T = 4096


def shared_blocks(shared: Sequence[Tuple[torch.Tensor, torch.Tensor]], f: int):
    """Cut always-on SwiGLU experts into experts of width f (every expert's width
    a multiple of f): expert u of width m f becomes m experts, block j taking gate
    rows [j f, (j+1) f), the matching up rows and the matching columns of W2.  The
    blocks' outputs sum to the expert's (SiLU(a) * b is taken per element of h, and
    the down product sums over h).  Returns (w13 blocks, w2 blocks), or None when
    some width is not a multiple of f."""
    if f < 1 or not shared:
        return None
    b13, b2 = [], []
    for w13, w2 in shared:
        fu = w13.shape[0] // 2
        if fu % f:
            return None
        for j in range(fu // f):
            b13.append(torch.cat([w13[j * f:(j + 1) * f], w13[fu + j * f:fu + (j + 1) * f]],
                                 0).contiguous())
            b2.append(w2[:, j * f:(j + 1) * f].contiguous())
    return b13, b2


def concat_shared(shared: Sequence[Tuple[torch.Tensor, torch.Tensor]]):
    """Lay several always-on SwiGLU experts out as one wider expert.

    For experts u with W13_u = [G_u; U_u] and W2_u, the sum over u of
    W2_u (SiLU(G_u x) * U_u x) equals the single expert with gate rows
    [G_0; G_1; ...], up rows [U_0; U_1; ...] and W2 = [W2_0 | W2_1 | ...].
    """
    if not shared:
        return None
    if len(shared) == 1:
        return shared[0][0].contiguous(), shared[0][1].contiguous()
    gates, ups, downs = [], [], []
    for w13, w2 in shared:
        f = w13.shape[0] // 2
        gates.append(w13[:f])
        ups.append(w13[f:])
        downs.append(w2)
    return torch.cat(gates + ups, 0).contiguous(), torch.cat(downs, 1).contiguous()


class LayerShare:
    def __init__(self, X: torch.Tensor, Wr: torch.Tensor, bias: Optional[torch.Tensor], k: int,
                 placement: np.ndarray, dev: int, w13: Sequence[torch.Tensor],
                 w2: Sequence[torch.Tensor], shared=(), renorm: bool = True,
                 coact: bool = False, want_logits: bool = True, cap_rows: Optional[int] = None,
                 gather_in_ffn: Optional[bool] = None, overlap_shared: bool = True,
                 fuse_combine: Optional[bool] = None, shared_in_ffn: Optional[bool] = None):
        self.device = X.device
        self.X = X
        self.Wr = Wr
        self.bias = bias
        self.T, self.d = X.shape
        self.E = Wr.shape[0]
        self.k = k
        self.dev = dev
        self.renorm = renorm
        self.want_coact = coact
        # gather_in_ffn: the permute step writes only the row maps and the expert
        # FFN reads its rows from X through row_token (moe_grouped_ffn_rows).  None:
        # for bf16 batches of at least 16384 token-expert assignments, where the row
        # copy it saves is large (measured faster at the DeepSeek-V2-Lite and Qwen3
        # prefill shapes, even at Mixtral's, slower at Qwen1.5's 8192), and for bf16
        # batches of at most 256 tokens, where the copy is a launch of its own for
        # little data (Qwen3-30B-A3B-shaped decode step 74.4 -> 71.3 us), unless
        # the share fuses the combine into the FFN call, which reads the packaged rows
        packaged_asked = gather_in_ffn is False
        if gather_in_ffn is None:
            fusable = fuse_combine is True or (fuse_combine is None and X.shape[0] <= 64 and k <= 2)
            gather_in_ffn = X.dtype == torch.bfloat16 and (
                X.shape[0] * k >= 16384 or (X.shape[0] <= 256 and not fusable))
        # shared_in_ffn: the shared experts as leading groups of the routed call (see
        # the module docstring), which reads its rows through row_token.  None: bf16
        # batches of at most SHARED_IN_FFN_MAX_T tokens whose shared experts' widths
        # are multiples of f, unless the packaged row copy was asked for
        # (gather_in_ffn=False)
        f_routed = w13[0].shape[0] // 2 if len(w13) else 0
        blocks = shared_blocks(list(shared), f_routed) if shared and shared_in_ffn is not False else None
        if shared_in_ffn is None:
            shared_in_ffn = (blocks is not None and X.dtype == torch.bfloat16
                             and 1 <= X.shape[0] <= SHARED_IN_FFN_MAX_T and not packaged_asked)
        if shared_in_ffn and blocks is None:
            raise ValueError("shared_in_ffn needs shared experts whose widths are multiples "
                             "of the routed experts' f")
        self.shared_in_ffn = bool(shared_in_ffn)
        self.n_shared_blocks = len(blocks[0]) if self.shared_in_ffn else 0
        # the leading groups read their rows through row_token
        if self.shared_in_ffn:
            gather_in_ffn = True
        self.gather_in_ffn = bool(gather_in_ffn)
        self.placement = np.ascontiguousarray(placement, dtype=np.uint8)
        self.G = self.placement.shape[1]
        self.n_local = int(self.placement[:, dev].sum())
        self.cap_rows = cap_rows if cap_rows is not None else self.T * min(k, self.n_local)
        T, d, E, dt = self.T, self.d, self.E, X.dtype
        dv = self.device
        self.logits = torch.empty((T, E), dtype=torch.float32, device=dv) if want_logits else None
        self.topk_idx = torch.empty((T, k), dtype=torch.int32, device=dv)
        self.topk_gate = torch.empty((T, k), dtype=torch.float32, device=dv)
        dcode = moe.MOE_BF16 if dt == torch.bfloat16 else moe.MOE_F32
        rb = moe.moe_route_topk_ws_bytes(dcode, T, d, E, moe.MOE_RENORM if renorm else 0)
        self.ws_route = moe.workspace(rb, dv) if rb else None
        self.counts = torch.empty((E,), dtype=torch.int32, device=dv)
        self.coact = torch.empty((E, E), dtype=torch.int32, device=dv) if coact else None
        cap = max(self.cap_rows, 1)
        # leading rows of the shared experts' blocks (shared_in_ffn): block j's rows
        # [j T, (j+1) T) are the tokens in order, ahead of the routed rows
        lead = self.n_shared_blocks * T
        self._row_token_all = torch.empty((lead + cap,), dtype=torch.int32, device=dv)
        if lead:
            self._row_token_all[:lead].copy_(
                torch.arange(T, dtype=torch.int32, device=dv).repeat(self.n_shared_blocks))
        self.perm = {
            "x_perm": None if gather_in_ffn else torch.empty((cap, d), dtype=dt, device=dv),
            "group_offsets": torch.empty((self.n_local + 1,), dtype=torch.int32, device=dv),
            "row_token": self._row_token_all[lead:],
            "row_gate": torch.empty((cap,), dtype=torch.float32, device=dv),
            "token_row": torch.empty((T, k), dtype=torch.int32, device=dv),
            "send_counts": torch.empty((self.G,), dtype=torch.int32, device=dv),
        }
        self.ws_perm = moe.workspace(moe.moe_permute_ws_bytes(T, k, E), dv)
        # y_perm: the routed rows (shared_in_ffn: after the shared blocks' slices)
        self._y_perm_all = torch.empty((lead + cap, d), dtype=dt, device=dv)
        self.y_perm = self._y_perm_all[lead:]
        self.y_shared_slices = self._y_perm_all[:lead] if lead else None
        self.weights = moe.WeightTable(w13, w2) if self.n_local else None
        self.f = self.weights.f if self.weights else f_routed
        dcode = moe.MOE_BF16 if dt == torch.bfloat16 else moe.MOE_F32
        self._blocks = blocks if self.shared_in_ffn else None
        self._ffn_weights = self._call_weights(w13, w2)
        self.ws_ffn = moe.workspace(
            moe.moe_grouped_ffn_ws_bytes(dcode, lead + self.cap_rows, d, max(self.f, 1),
                                         max(self.n_shared_blocks + self.n_local, 1)), dv)
        sh = concat_shared(list(shared)) if not self.shared_in_ffn else None
        if sh is not None:
            self.shared_weights = moe.WeightTable([sh[0]], [sh[1]])
            self.shared_offsets = torch.tensor([0, T], dtype=torch.int32, device=dv)
            self.y_shared = torch.empty((max(T, 1), d), dtype=dt, device=dv)
            self.ws_shared = moe.workspace(
                moe.moe_grouped_ffn_ws_bytes(dcode, T, d, self.shared_weights.f, 1), dv)
        else:
            self.shared_weights = None
            self.y_shared = None
        # second stream for the shared experts (default priority), fork/join events
        self._side = None
        if self.shared_weights is not None and overlap_shared:
            self._side = torch.cuda.Stream(device=dv)
            self._fork = torch.cuda.Event(enable_timing=False)
            self._join = torch.cuda.Event(enable_timing=False)
        self.y = torch.empty((max(T, 1), d), dtype=dt, device=dv)
        # a token reaches an expert at most once, so with at most 256 tokens no group
        # exceeds the streaming kernels' limit; when the mean group is decode-sized
        # (T k / E <= 64 rows) every group is streamed and the tiled launches are
        # left out (the shared experts' call, one group of T rows, likewise)
        self.ffn_products = moe.MOE_FFN_GATE_UP | moe.MOE_FFN_DOWN
        if T <= 64 or (T <= 256 and T * k <= 64 * self.E):
            self.ffn_products |= moe.MOE_FFN_SMALL_GROUPS
        # with the shared blocks in the call, over more than 256 tokens they make
        # enough tiles that no group is streamed: the streaming launches are left
        # out (a hint only: the routed groups are tiled whatever their size)
        elif self.shared_in_ffn and T > 256:
            self.ffn_products |= moe.MOE_FFN_LARGE_GROUPS
        # when the mean group is at least 512 rows, a call short enough to stream its
        # groups (at most a quarter of the CUs' worth of tiles in its groups above 64
        # rows) would need this GPU's experts to get a small fraction of their share:
        # every group is tiled and the streaming launches, which would find nothing to
        # do, are left out (a hint only: any group sizes give correct results)
        elif T * k >= 512 * self.E:
            self.ffn_products |= moe.MOE_FFN_LARGE_GROUPS
        # ... and then the combine can run inside the down product's chunk sum
        # (moe_grouped_ffn_combine: y_perm is not written).  fuse_combine None: where
        # it measured faster, batches of at most 64 tokens with k <= 2 (at k = 6 or 8
        # the fused chunk sum, k x S partial loads per output element, is slower than
        # the chunk sum plus the combine launch); True: whenever the call streams
        # every group; False: never
        # the shared experts' call is one group of T rows: above 256 rows it is tiled
        # whole and its streaming launches are left out (MOE_FFN_LARGE_GROUPS)
        self.shared_products = self.ffn_products & ~moe.MOE_FFN_LARGE_GROUPS
        if T > 256:
            self.shared_products |= moe.MOE_FFN_LARGE_GROUPS
        can_fuse = (bool(self.ffn_products & moe.MOE_FFN_SMALL_GROUPS) and dt == torch.bfloat16
                    and not gather_in_ffn and self.weights is not None
                    and not self.shared_in_ffn)
        if fuse_combine is None:
            fuse_combine = T <= 64 and k <= 2
        self.fused_combine = bool(fuse_combine) and can_fuse

    def set_placement(self, placement: np.ndarray, w13: Sequence[torch.Tensor],
                      w2: Sequence[torch.Tensor]):
        """Swap the expert placement between batches (same number of local slots)."""
        placement = np.ascontiguousarray(placement, dtype=np.uint8)
        n_local = int(placement[:, self.dev].sum())
        if n_local != self.n_local:
            raise ValueError("the new placement must keep %d local slots" % self.n_local)
        self.placement = placement
        self.weights = moe.WeightTable(w13, w2)
        self._ffn_weights = self._call_weights(w13, w2)

    def _call_weights(self, w13: Sequence[torch.Tensor], w2: Sequence[torch.Tensor]):
        """The weight table of the FFN call: the routed experts', led by the shared
        blocks' when they share the call."""
        if not self.shared_in_ffn:
            return self.weights
        w13 = list(w13)[:self.n_local]
        w2 = list(w2)[:self.n_local]
        return moe.WeightTable(self._blocks[0] + w13, self._blocks[1] + w2)

    def set_inputs(self, X: torch.Tensor, bias: Optional[torch.Tensor] = None):
        if tuple(X.shape) != (self.T, self.d) or X.dtype != self.X.dtype:
            raise ValueError("X must keep shape and dtype")
        self.X = X
        if bias is not None:
            self.bias = bias

    def route(self, logits_in: Optional[torch.Tensor] = None):
        if logits_in is not None:
            moe.moe_route_topk(None, None, None, self.k, renorm=self.renorm, logits=logits_in,
                               logits_in=True, topk_idx=self.topk_idx, topk_gate=self.topk_gate)
        else:
            moe.moe_route_topk(self.X, self.Wr, self.bias, self.k, renorm=self.renorm,
                               logits=self.logits, want_logits=self.logits is not None,
                               topk_idx=self.topk_idx, topk_gate=self.topk_gate, ws=self.ws_route)

    def _shared_ffn(self, stream=None):
        """The shared experts' call of their own (nothing when they share the routed
        call, or there are none)."""
        if self.shared_weights is None:
            return
        moe.moe_grouped_ffn(self.X, self.shared_offsets, self.shared_weights, cap_rows=self.T,
                            y_perm=self.y_shared, ws=self.ws_shared, stream=stream,
                            products=self.shared_products)

    def combine(self):
        """Enqueue the combine as `run` makes it (after the FFN call or calls)."""
        if self.shared_in_ffn:
            moe.moe_combine_shared(self.y_perm, self.perm["token_row"], self.topk_gate,
                                   self.y_shared_slices, self.n_shared_blocks, T=self.T, d=self.d,
                                   y=self.y)
        else:
            moe.moe_combine(self.y_perm, self.perm["token_row"], self.topk_gate, self.y_shared,
                            T=self.T, d=self.d, y=self.y)

    def shared_output(self) -> Optional[torch.Tensor]:
        """The shared experts' output [T, d] in fp32 (the blocks' slices summed in
        order when they share the routed call), for checks; None without shared
        experts.  Valid once the step has completed."""
        if self.shared_in_ffn:
            sl = self.y_shared_slices.view(self.n_shared_blocks, self.T, self.d).float()
            out = sl[0].clone()
            for j in range(1, self.n_shared_blocks):
                out += sl[j]
            return out
        return None if self.y_shared is None else self.y_shared[:self.T].float()

    def package(self):
        """Enqueue the packaging step as `run` makes it (moe_permute; the row copy
        x_perm only when the FFN does not gather the rows itself)."""
        moe.moe_permute(self.X, self.topk_idx, self.topk_gate, self.counts, self.placement,
                        self.dev, E=self.E, cap_rows=self.cap_rows, out=self.perm, ws=self.ws_perm,
                        copy_rows=not self.gather_in_ffn)

    def routed_ffn(self, fused: Optional[bool] = None):
        """Enqueue the routed experts' FFN call as `run` makes it: moe_grouped_ffn (or
        moe_grouped_ffn_rows) into y_perm, or, when the share fuses the combine (fused
        None: as `run` does), moe_grouped_ffn_combine into y (which then reads y_shared:
        the shared experts' call must have completed on this stream)."""
        if self.shared_in_ffn:
            moe.moe_grouped_ffn_rows_shared(self.X, self._row_token_all, self.perm["group_offsets"],
                                            self._ffn_weights, self.n_shared_blocks,
                                            cap_rows=self.cap_rows, y_perm=self._y_perm_all,
                                            ws=self.ws_ffn, products=self.ffn_products)
            return
        if self.weights is None:
            return
        if self.fused_combine if fused is None else (fused and self.fused_combine):
            moe.moe_grouped_ffn_combine(self.perm["x_perm"], self.perm["group_offsets"],
                                        self.weights, self.perm["token_row"], self.topk_gate,
                                        self.y_shared, cap_rows=self.cap_rows, T=self.T, y=self.y,
                                        ws=self.ws_ffn)
        elif self.gather_in_ffn:
            moe.moe_grouped_ffn_rows(self.X, self.perm["row_token"], self.perm["group_offsets"],
                                     self.weights, cap_rows=self.cap_rows, y_perm=self.y_perm,
                                     ws=self.ws_ffn, products=self.ffn_products)
        else:
            moe.moe_grouped_ffn(self.perm["x_perm"], self.perm["group_offsets"], self.weights,
                                cap_rows=self.cap_rows, y_perm=self.y_perm, ws=self.ws_ffn,
                                products=self.ffn_products)

    def run(self, logits_in: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Enqueue the whole share after the current stream's earlier work; returns y
        [T, d], complete on the current stream (the shared experts' branch, if
        any, is joined back before the combine)."""
        main = torch.cuda.current_stream(self.device)

        def fork_shared():
            self._fork.record(main)
            self._side.wait_event(self._fork)
            self._shared_ffn(self._side)
            self._join.record(self._side)

        if self.fused_combine:
            # the fused call reads y_shared: the shared branch overlaps the routing
            if self._side is not None:
                fork_shared()
            self.route(logits_in)
            moe.moe_expert_histogram(self.topk_idx, self.E, counts=self.counts, coact=self.coact)
            self.package()
            if self._side is not None:
                main.wait_event(self._join)
            elif self.shared_weights is not None:
                self._shared_ffn()
            self.routed_ffn()
            return self.y
        self.route(logits_in)
        moe.moe_expert_histogram(self.topk_idx, self.E, counts=self.counts, coact=self.coact)
        self.package()
        # the shared branch forks after the routing launches, which would otherwise
        # wait for CUs held by its GEMMs, and overlaps the routed experts' FFN, whose
        # launches leave CUs idle
        if self._side is not None:
            fork_shared()
        self.routed_ffn()
        if self._side is not None:
            main.wait_event(self._join)
        else:
            self._shared_ffn()
        self.combine()
        return self.y
