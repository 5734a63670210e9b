"""One worker replica's synchronous SGD step, driven through the tfk_* ops.

The schedule follows the paper's single-replica semantics (Sections 4.1 and
4.4): a forward pass over every op (each convolution with its bias and ReLU
fused into one kernel, Section 5); the upstream gradient ``g`` of the output
tensor seeds a backward pass that visits the ops in reverse order and sums the
partial gradients of every path into a tensor (``beta = 1`` for every
contribution after the first); no gradient is formed for the step input
unless the workload asks for it; then every variable is updated in place with
W' = W - lr * dW, all from gradients computed with the same pre-update
parameters.

Memory layout (all on one GPU):

* Variables: one flat fp32 buffer holding every filter (HWIO) and bias, each
  at a 256-byte aligned offset, and a flat fp32 gradient buffer with the same
  layout, so the whole update is one ApplyGradientDescent launch.  For bf16
  workloads a flat bf16 shadow of the variables (written by that same launch)
  holds the filters the convolutions read.
* Activations: one NHWC buffer per tensor in the workload's storage type.
  Inception concat buffers are written by their branches as channel slices
  and read back the same way, so no concat or split is ever copied.
* Gradients: one NHWC buffer per tensor (ReLU-backward writes its result over
  the incoming gradient, except for the seed ``g`` which stays intact).

A max-pool whose input is the whole output of one convolution and is read by
nothing else runs its backward fused with that convolution's ReLU backward and
bias gradient (one kernel writes dL/d(pre-activation) directly, Section 5's
fused activation gradients); that convolution then skips its own ReLU backward.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import ops
from .workloads import Conv, Inputs, Net, Pool

_ALIGN = 64   # elements: 256 bytes of fp32


def _align(n: int) -> int:
    return (n + _ALIGN - 1) // _ALIGN * _ALIGN


def _merge_groups(net: Net):
    """1x1 convolutions (stride 1, ReLU) that read one tensor, at least two of them, each writing
    either a tensor of its own or the first channels of a concat tensor (at most one per group).
    Their outputs are laid out side by side in one buffer -- the own tensors first, then the concat
    whose first channels that one writes -- so that one convolution with their filters side by side
    (a wider 1x1) computes them all: one pass over the input per direction instead of one per
    member (an inception module's branch reductions)."""
    if net.dtype != "bf16":
        return []
    writers = {}
    for op in net.ops:
        writers.setdefault(op.dst, []).append(op)
    pos = {op.name: k for k, op in enumerate(net.ops)}
    cand = {}
    for c in net.convs:
        if not (c.kh == c.kw == 1 and c.sh == c.sw == 1 and tuple(c.pads) == (0, 0, 0, 0) and c.relu):
            continue
        if c.dst in ("x", net.output):
            continue
        k = pos[c.name]
        nxt = net.ops[k + 1] if k + 1 < len(net.ops) else None
        if isinstance(nxt, Pool) and nxt.src == c.dst:
            continue                                  # (its forward runs with that pool)
        cand.setdefault(c.src, []).append(c)
    groups, used = [], set()
    for src, cs in cand.items():
        own = [c for c in cs if c.dst_c0 == 0 and c.cout == net.tensors[c.dst][3] and writers[c.dst] == [c]
               and c.dst not in used]
        cat = [c for c in cs if c not in own and c.dst_c0 == 0 and c.dst not in used]
        members = own + cat[:1]
        if len(members) < 2:
            continue
        offs, w = {}, 0
        for c in own:
            offs[c.dst] = w
            w += c.cout
        catt = cat[0].dst if cat else None
        if catt is not None:
            offs[catt] = w
            w += net.tensors[catt][3]
        used.update(offs)
        first = min(members, key=lambda c: pos[c.name])
        mconv = Conv(name="merged_" + first.name, src=src, dst="merged_" + first.name, dst_c0=0,
                     cout=sum(c.cout for c in members), kh=1, kw=1, sh=1, sw=1, pads=(0, 0, 0, 0))
        groups.append({"op": mconv, "members": members, "offs": offs, "width": w, "cat": catt,
                       "at": pos[first.name]})
    return groups


def access_deps(reads, writes, ordered_writes=True):
    """For ops in issue order with the tensor names each reads and writes, the earlier ops each
    must follow: a read after a write, a write after a read, and, with ``ordered_writes``, a
    write after a write (gradient accumulation keeps its order; the forward pass's writers of
    one concat write disjoint channel slices and need no order)."""
    deps = []
    for i in range(len(reads)):
        deps.append([j for j in range(i) if (writes[j] & reads[i]) or (reads[j] & writes[i])
                     or (ordered_writes and (writes[j] & writes[i]))])
    return deps


def lane_plan(nodes, deps, nlanes: int):
    """Places ops, in issue order, on ``nlanes`` streams: an op continues the lane of a producer
    it needs when that producer is the lane's latest op, else takes the least recently used lane,
    so an inception module's branches run side by side.  ``deps[i]`` lists the earlier ops node i
    must follow (see access_deps).  Returns ``(plan, joins)``: plan entries ``(op, lane, waits)``,
    ``waits`` the earlier nodes (by index) on other lanes whose completion the op needs and its
    lane has not yet waited for, directly or through another wait (vector clocks), at most one
    per lane; "start" is lane 0 at the start, which every lane's first op must follow.
    ``joins`` are the nodes lane 0 waits for at the end, so that it follows every node."""
    lane_of: List[int] = []
    tail = [None] * nlanes                   # latest node of each lane
    used_at = [-1] * nlanes                  # when each lane was last given a node
    clock = [dict() for _ in range(nlanes)]  # lane -> {lane: latest node known complete}
    clock[0][0] = -1                         # lane 0 starts where the caller's stream is
    node_clock, plan = [], []
    for i, op in enumerate(nodes):
        need = sorted(deps[i])
        cont = [lane_of[j] for j in need if tail[lane_of[j]] == j]
        if i == 0:
            lane = 0
        elif cont:
            lane = 0 if 0 in cont else cont[-1]
        else:
            lane = min(range(nlanes), key=lambda k: used_at[k])
        waits = []
        c = clock[lane]
        latest = {}                          # per producing lane, its latest node among deps
        for j in need:
            latest[lane_of[j]] = max(latest.get(lane_of[j], -1), j)
        for a, j in sorted(latest.items(), key=lambda t: t[1]):
            if a != lane and c.get(a, -2) < j:
                waits.append(j)
                for k, v in node_clock[j].items():
                    c[k] = max(c.get(k, -2), v)
        if c.get(0, -2) < -1:
            waits.insert(0, "start")
            c[0] = -1
        c[lane] = i
        lane_of.append(lane)
        tail[lane] = i
        used_at[lane] = i
        node_clock.append(dict(c))
        plan.append((op, lane, waits))
    joins = []
    for k in range(1, nlanes):
        if tail[k] is not None and clock[0].get(k, -2) < tail[k]:
            joins.append(tail[k])
            for kk, v in node_clock[tail[k]].items():
                clock[0][kk] = max(clock[0].get(kk, -2), v)
    return plan, joins


class Replica:
    """Device state of one replica of ``net`` and its training step."""

    def __init__(self, net: Net, inputs: Inputs, device: str = "cuda", optimizer: str = "sgd",
                 momentum: float = 0.9, nesterov: bool = False, beta1: float = 0.9, beta2: float = 0.999,
                 epsilon: float = 1e-8, merge: bool = True):
        """``optimizer`` picks the in-place variable update that ends the step: "sgd"
        (ApplyGradientDescent), "momentum" (velocity slot, optional look-ahead form) or "adam"
        (two moment slots, bias-corrected by the step count).  ``merge``: run each group of 1x1
        convolutions that read one tensor as one wider convolution (see _merge_groups)."""
        if optimizer not in ("sgd", "momentum", "adam"):
            raise ValueError("optimizer is 'sgd', 'momentum' or 'adam'")
        self.net = net
        self.optimizer = optimizer
        self.opt_args = dict(momentum=momentum, nesterov=bool(nesterov), beta1=beta1, beta2=beta2, epsilon=epsilon)
        self.t = 0
        self.device = torch.device(device)
        self.dtype = torch.float32 if net.dtype == "f32" else torch.bfloat16
        self.lr = float(np.float32(net.lr))
        dev, dt = self.device, self.dtype

        # ---- 1x1 convolutions merged into one (their outputs side by side in one buffer)
        self.merges = _merge_groups(net) if merge else []
        member_of = {c.name: g for g in self.merges for c in g["members"]}
        store = {}                                   # tensor -> (storage name, first channel)
        for g in self.merges:
            for t, o in g["offs"].items():
                store[t] = (g["op"].name, o)

        # ---- variables
        # Filters first (a merged group's filters side by side as one HWIO block); then the
        # biases, in the channel order of the buffers the convolutions write (a concat's
        # branches, a merged group's members), so that a group of them has one contiguous
        # bias(-gradient) slice (see relu_groups and merges).
        off = 0
        self._layout = {}
        self._wslot = {}                             # name -> (block offset, block shape, first channel)
        for c in net.convs:
            g = member_of.get(c.name)
            if g is not None and g["op"].name in self._wslot:
                continue
            cin = net.tensors[c.src][3]
            cout = g["op"].cout if g is not None else c.cout
            key = g["op"].name if g is not None else c.name
            self._wslot[key] = (off, (c.kh, c.kw, cin, cout), 0)
            off += _align(c.kh * c.kw * cin * cout)
        for g in self.merges:
            bo, shp, _ = self._wslot[g["op"].name]
            a = 0
            for c in g["members"]:
                self._wslot[c.name] = (bo, shp, a)
                a += c.cout
        by_store = {}
        for c in net.convs:
            st, base = store.get(c.dst, (c.dst, 0))
            by_store.setdefault(st, []).append((base + c.dst_c0, c))
        for st, cs in by_store.items():
            off = _align(off)
            for _, c in sorted(cs, key=lambda e: e[0]):
                wo, wshape, a = self._wslot[c.name]
                self._layout[c.name] = (wo, wshape, off, c.cout)
                off += c.cout
        off = _align(off)
        self.n_params = off
        self.params = torch.zeros(off, dtype=torch.float32, device=dev)
        self.grads = torch.zeros(off, dtype=torch.float32, device=dev)
        self.shadow = torch.zeros(off, dtype=torch.bfloat16, device=dev) if dt == torch.bfloat16 else None
        # optimizer slots (zero at the start of training), laid out like params
        n_slots = {"sgd": 0, "momentum": 1, "adam": 2}[optimizer]
        self.slots = [torch.zeros(off, dtype=torch.float32, device=dev) for _ in range(n_slots)]
        host = np.zeros(off, dtype=np.float32)
        for c in net.convs:
            self.place_filter(host, c.name, inputs.weights[c.name])
            wo, wshape, bo, bn = self._layout[c.name]
            host[bo:bo + bn] = inputs.biases[c.name].astype(np.float32)
        p = torch.from_numpy(host)
        if dt == torch.bfloat16:
            p = p.to(torch.bfloat16).to(torch.float32)      # master weights start at the bf16 values
        self.params.copy_(p.to(dev))
        if self.shadow is not None:
            self.shadow.copy_(self.params.to(torch.bfloat16))
        self.W, self.b, self.dW, self.db, self.Wlp = {}, {}, {}, {}, {}
        blocks = {}
        for key, (wo, wshape, a) in self._wslot.items():
            if a == 0 and key not in member_of:
                wn = int(np.prod(wshape))
                blocks[key] = (self.params[wo:wo + wn].view(wshape), self.grads[wo:wo + wn].view(wshape),
                               self.shadow[wo:wo + wn].view(wshape) if self.shadow is not None else None)
        for c in net.convs:
            g = member_of.get(c.name)
            wo, wshape, a = self._wslot[c.name]
            W, dW, Wlp = blocks[g["op"].name if g is not None else c.name]
            sl = (Ellipsis, slice(a, a + c.cout))
            self.W[c.name], self.dW[c.name] = W[sl], dW[sl]
            self.Wlp[c.name] = Wlp[sl] if Wlp is not None else self.W[c.name]
            _, _, bo, bn = self._layout[c.name]
            self.b[c.name] = self.params[bo:bo + bn]
            self.db[c.name] = self.grads[bo:bo + bn]
        # the merged convolutions' dense filters and contiguous biases
        self.mW, self.mWlp, self.mdW, self.mb, self.mdb = {}, {}, {}, {}, {}
        for g in self.merges:
            name = g["op"].name
            W, dW, Wlp = blocks[name]
            self.mW[name], self.mdW[name] = W, dW
            self.mWlp[name] = Wlp if Wlp is not None else W
            bo = self._layout[g["members"][0].name][2]
            self.mb[name] = self.params[bo:bo + g["op"].cout]
            self.mdb[name] = self.grads[bo:bo + g["op"].cout]

        # ---- activations, gradients, argmax
        self.act: Dict[str, torch.Tensor] = {}
        for name, shape in net.tensors.items():
            if name == "x":
                xin = torch.from_numpy(inputs.x).to(dt).to(dev)
                if dt == torch.bfloat16 and shape[3] == 3:
                    # RGB images are kept as RGBx (a zero fourth channel): the first
                    # convolution reads them in place instead of padding them per call
                    buf = torch.zeros(shape[:3] + (4,), dtype=dt, device=dev)
                    buf[..., :3].copy_(xin)
                    xin = buf[..., :3]
                self.act["x"] = xin
            else:
                self.act[name] = torch.zeros(shape, dtype=dt, device=dev)
        if net.loss == "softmax_xent":
            # the logits' gradient is written by the cross-entropy kernel every step
            self.g = torch.zeros(net.tensors[net.output], dtype=dt, device=dev)
            self.labels = torch.from_numpy(np.asarray(inputs.labels, dtype=np.int32)).to(dev)
            self.loss_rows = torch.zeros(self.labels.numel(), dtype=torch.float32, device=dev)
        else:
            self.g = torch.from_numpy(inputs.g).to(dt).to(dev)
        self.grad: Dict[str, torch.Tensor] = {net.output: self.g}
        for name, shape in net.tensors.items():
            if name == net.output or (name == "x" and not net.input_grad):
                continue
            self.grad[name] = torch.zeros(shape, dtype=dt, device=dev)
        # merged groups: one buffer each for the activations and one for the gradients, the
        # members' tensors (and the concat) channel slices of it
        self.m_act, self.m_grad = {}, {}
        for g in self.merges:
            shape = net.tensors[g["members"][0].dst][:3] + (g["width"],)
            A = torch.zeros(shape, dtype=dt, device=dev)
            G = torch.zeros(shape, dtype=dt, device=dev)
            for t, o in g["offs"].items():
                w = net.tensors[t][3]
                self.act[t] = A[..., o:o + w]
                self.grad[t] = G[..., o:o + w]
            self.m_act[g["op"].name] = A[..., :g["op"].cout]
            self.m_grad[g["op"].name] = G[..., :g["op"].cout]
        # the ops the step runs: each merged group's members replaced by its convolution, at the
        # place of its first member
        merged_at = {g["at"]: g["op"] for g in self.merges}
        self.ops = []
        for k, op in enumerate(net.ops):
            if k in merged_at:
                self.ops.append(merged_at[k])
            if op.name not in member_of:
                self.ops.append(op)
        self.merged = {g["op"].name: g for g in self.merges}
        # ReLU-backward of the ops that write the output tensor must not overwrite the seed g
        self.dpre_out = torch.zeros(net.tensors[net.output], dtype=dt, device=dev)
        # each max-pool's selection as uint8 window taps (windows of at most 256 taps)
        self.argmax = {op.name: torch.zeros(net.tensors[op.dst][:3] + (net.tensors[op.src][3],),
                                            dtype=torch.uint8 if op.kh * op.kw <= 256 else torch.int32,
                                            device=dev)
                       for op in net.ops if isinstance(op, Pool)}
        # ---- max-pools fused with the ReLU backward of the convolution that feeds them
        writers, readers = {}, {}
        for op in net.ops:
            writers.setdefault(op.dst, []).append(op)
            readers.setdefault(op.src, []).append(op)
        self.pool_relu = {}                      # pool name -> conv
        for op in net.ops:
            if isinstance(op, Pool):
                w = writers.get(op.src, [])
                if (len(w) == 1 and isinstance(w[0], Conv) and w[0].relu and w[0].dst_c0 == 0
                        and w[0].cout == net.tensors[op.src][3] and len(readers[op.src]) == 1):
                    self.pool_relu[op.name] = w[0]
        # ---- convolutions whose input is the whole ReLU output of another convolution and
        # feeds nothing else: their input gradient applies that ReLU backward in its epilogue
        self.bwi_relu = {}                       # conv name -> the conv that produced its input
        for op in net.ops:
            if isinstance(op, Conv) and op.src != "x" and op.src != net.output:
                w = writers.get(op.src, [])
                if (len(w) == 1 and isinstance(w[0], Conv) and w[0].relu and w[0].dst_c0 == 0
                        and w[0].cout == net.tensors[op.src][3] and len(readers[op.src]) == 1):
                    self.bwi_relu[op.name] = w[0]
        self.relu_fused = ({c.name for c in self.pool_relu.values()} |
                           {c.name for c in self.bwi_relu.values()})
        # ---- convolutions writing adjacent channel ranges of one tensor (a concat's branches,
        # each with its own ReLU and bias) whose readers all come after the last of them: their
        # ReLU backward runs once over the whole range, with one bias-gradient reduction into
        # their adjacent bias-gradient slices
        pos = {op.name: k for k, op in enumerate(net.ops)}
        by_dst = {}
        for c in net.convs:
            by_dst.setdefault(c.dst, []).append(c)
        self.relu_groups = {}                    # conv name -> (first channel, width, [convs])
        for dst, cs in by_dst.items():
            cand = sorted((c for c in cs if c.relu and c.name not in self.relu_fused and dst != net.output),
                          key=lambda c: c.dst_c0)
            runs, cur = [], []
            for c in cand:
                if cur and c.dst_c0 == cur[-1].dst_c0 + cur[-1].cout:
                    cur.append(c)
                else:
                    if len(cur) > 1:
                        runs.append(cur)
                    cur = [c]
            if len(cur) > 1:
                runs.append(cur)
            for run in runs:
                last = max(pos[c.name] for c in run)
                if all(pos[r.name] > last for r in readers.get(dst, [])):
                    g = (run[0].dst_c0, sum(c.cout for c in run), run)
                    for c in run:
                        self.relu_groups[c.name] = g
        # ---- a ReLU group over a whole tensor (a concat's branches) is applied by the last of the
        # tensor's readers to write its gradient (the first in forward order): a convolution's
        # input gradient, or a max-pool's, adds its part to what the others stored and masks and
        # sums the bias gradient in the same pass (no separate ReLU-backward pass over the concat)
        self.relu_last = {}                      # reader op name -> (tensor, group)
        for t, g in {run[0].dst: (c0, width, run) for c0, width, run in self.relu_groups.values()}.items():
            c0, width, run = g
            if c0 != 0 or width != net.tensors[t][3] or t in ("x", net.output):
                continue
            first = next((op for op in self.ops if op.src == t), None)
            if first is None or (isinstance(first, Conv) and first.name in self.bwi_relu):
                continue
            if isinstance(first, Pool) and first.name in self.pool_relu:
                continue
            self.relu_last[first.name] = (t, g)
        # ---- a convolution whose whole ReLU output is pooled by the next op: one forward call
        # (one kernel where its row bands hold whole pool windows)
        self.conv_pool = {}                      # conv name -> pool op
        for k, op in enumerate(net.ops[:-1]):
            nxt = net.ops[k + 1]
            if (isinstance(op, Conv) and op.relu and isinstance(nxt, Pool) and nxt.src == op.dst
                    and op.dst_c0 == 0 and op.cout == net.tensors[op.dst][3] and writers[op.dst] == [op]
                    and self.argmax[nxt.name].dtype == torch.uint8):
                self.conv_pool[op.name] = nxt
        self.pool_in_conv = {p.name for p in self.conv_pool.values()}
        # ---- one workspace big enough for every op
        need = 0
        for c in net.convs:
            x = self.act[c.src]
            for op_kind in (0, 1, 2, 3) if c.name in self.bwi_relu else (0, 1, 2):
                need = max(need, ops.conv2d_workspace_bytes(op_kind, x, c.cout, c.kh, c.kw, (c.sh, c.sw), c.pads))
            need = max(need, ops.bias_relu_bwd_workspace_bytes(self._slice(self.act, c)))
        for c0, width, run in {id(g[2]): g for g in self.relu_groups.values()}.values():
            need = max(need, ops.bias_relu_bwd_workspace_bytes(self.act[run[0].dst][..., c0:c0 + width]))
        for g in self.merges:
            m = g["op"]
            for op_kind in (0, 1):
                need = max(need, ops.conv2d_workspace_bytes(op_kind, self.act[m.src], m.cout, 1, 1, (1, 1), m.pads))
        self.ws = torch.zeros(max(16, (need + 15) // 16 * 16), dtype=torch.uint8, device=dev)
        # ---- filter gradients run on a second stream, with a workspace of their own
        need = 0
        for c in list(net.convs) + [g["op"] for g in self.merges]:
            need = max(need, ops.conv2d_workspace_bytes(2, self.act[c.src], c.cout, c.kh, c.kw, (c.sh, c.sw),
                                                        c.pads))
        self.ws_side = torch.zeros(max(16, (need + 15) // 16 * 16), dtype=torch.uint8, device=dev)
        self.side = torch.cuda.Stream(device=dev)
        # ---- the forward pass's independent branches run on up to kFwdLanes streams (lane 0 is
        # the step's stream, lane 1 the side stream, idle in the forward pass: with the step's
        # stream, four streams, as many as the hardware queues a process gets by default), each
        # lane with a workspace of its own (see _forward_plan)
        self.fwd_plan = self._forward_plan(self.kFwdLanes)
        # ---- the backward pass's independent branches: kBwdLanes streams (the side stream carries
        # the filter gradients there); backward lane k runs on lane stream k + 1
        self.bwd_plan = self._backward_plan(self.kBwdLanes)
        used = sorted(({lane for _, lane, _ in self.fwd_plan[0]} | {lane + 1 for _, lane, _ in self.bwd_plan[0]
                                                                    if lane > 0}) - {0})
        self.lane_streams = {k: self.side if k == 1 else torch.cuda.Stream(device=dev) for k in used}
        self.lane_ws = {k: torch.zeros_like(self.ws) for k in used}
        self.marks = {}                          # node index (or "start") -> ops.Mark, made on first use
        # ---- bias gradients of an untraced step: each ReLU/bias backward leaves its per-block
        # partials in a workspace of its own, and one launch sums them all before the update
        self.defer_bias = True
        self.bias_ws: Dict[object, torch.Tensor] = {}

    # ------------------------------------------------------------------ helpers
    # lanes of the forward and backward passes (sustained program steps, forward / backward:
    # 4 / 3 GoogLeNet 2.96-2.97 ms, Inception-v3 4.52; 4 / 2 2.95 and 4.48-4.50; 4 / 1 3.03 and
    # 4.56; 3 / 2 2.93 and 5.33, where a three-stream forward lines Inception's branches up badly)
    kFwdLanes = 4
    kBwdLanes = 2

    def _forward_plan(self, nlanes: int):
        """The forward ops (a pool made inside its convolution left out) placed on ``nlanes``
        streams by ``lane_plan``."""
        nodes, outs = [], []
        for op in self.ops:
            if isinstance(op, Pool) and op.name in self.pool_in_conv:
                continue
            if op.name in self.merged:
                o = {m.dst for m in self.merged[op.name]["members"]}
            elif op.name in self.conv_pool:
                o = {op.dst, self.conv_pool[op.name].dst}
            else:
                o = {op.dst}
            nodes.append(op)
            outs.append(o)
        return lane_plan(nodes, access_deps([{op.src} for op in nodes], outs, ordered_writes=False), nlanes)

    def _backward_access(self):
        """The backward nodes (reverse forward order) with the gradient tensors each reads and
        writes: its output gradient (read; written too where its ReLU or bias backward runs in
        place, which a concat's ReLU group does in its first node unless the concat's last
        reader has done it) and its input's gradient (written, accumulated after earlier
        writers)."""
        net, grouped = self.net, set()
        nodes, reads, writes = [], [], []
        for op in reversed(self.ops):
            src_grad = op.src != "x" or net.input_grad
            r, w = set(), set()
            if isinstance(op, Pool):
                r.add(op.dst)
                if op.name in self.pool_relu or src_grad:
                    w.add(op.src)
                if src_grad and op.name in self.relu_last:
                    grouped.add(id(self.relu_last[op.name][1][2]))
            else:
                members = self.merged[op.name]["members"] if op.name in self.merged else [op]
                for m in members:
                    r.add(m.dst)
                    if not m.relu or (m.name not in self.relu_fused and m.name not in self.relu_groups):
                        # (the output's pre-activation gradient: a buffer slice of this op's own)
                        w.add(m.dst if m.dst != net.output else "dpre_out:" + m.name)
                    elif m.name in self.relu_groups and id(self.relu_groups[m.name][2]) not in grouped:
                        grouped.add(id(self.relu_groups[m.name][2]))
                        w.add(m.dst)
                if src_grad:
                    w.add(op.src)
                    if op.name in self.relu_last:
                        grouped.add(id(self.relu_last[op.name][1][2]))
            nodes.append(op)
            reads.append(r)
            writes.append(w)
        return nodes, reads, writes

    def _backward_plan(self, nlanes: int):
        nodes, reads, writes = self._backward_access()
        return lane_plan(nodes, access_deps(reads, writes), nlanes)

    def _mark(self, key):
        m = self.marks.get(key)
        if m is None:
            m = self.marks[key] = ops.Mark()
        return m

    def place_filter(self, flat, name: str, w) -> None:
        """Writes filter ``w`` (HWIO) of convolution ``name`` where the flat variable layout keeps
        it: its own block, or its channels of its merged group's block."""
        wo, (kh, kw, cin, cout), a = self._wslot[name]
        blk = flat[wo:wo + kh * kw * cin * cout].reshape(kh, kw, cin, cout)
        blk[..., a:a + w.shape[3]] = w

    def _bias_ws(self, key, need: int) -> torch.Tensor:
        """The workspace of one deferred bias gradient, made at its first use and kept (a recorded
        program finds its partials where its calls left them).  Left uninitialised: its producer
        writes every partial it sums, and a fill on the allocating stream could land after a
        producer on a lane stream has written it."""
        t = self.bias_ws.get(key)
        if t is None or t.numel() < need:
            t = torch.empty(max(16, (need + 15) // 16 * 16), dtype=torch.uint8, device=self.params.device)
            self.bias_ws[key] = t
        return t

    def _width(self, op) -> int:
        return op.cout if isinstance(op, Conv) else self.net.tensors[op.src][3]

    def _slice(self, bufs, op):
        t = bufs[op.dst]
        return t[..., op.dst_c0:op.dst_c0 + self._width(op)]

    # ------------------------------------------------------------------ the step
    def forward(self, trace=None, stream=None, lanes=True):
        """The forward pass on ``stream``; untraced, with ``lanes``, independent branches run on
        the lane streams of the forward plan, which join ``stream`` before the loss."""
        if trace is not None or not lanes or not self.lane_streams or torch.cuda.is_current_stream_capturing():
            # (under HIP stream capture the forward pass stays on one stream: the marks are
            # persistent events, which are not recorded into captures)
            for op in self.ops:
                self._forward_op(op, trace, stream, self.ws)
        else:
            cur = stream if stream is not None else torch.cuda.current_stream()
            plan, joins = self.fwd_plan
            needed = {j for _, _, waits in plan for j in waits} | set(joins)
            if "start" in needed:
                self._mark("start").record(cur)
            for i, (op, lane, waits) in enumerate(plan):
                st = cur if lane == 0 else self.lane_streams[lane]
                for j in waits:
                    self._mark(j).wait(st)
                self._forward_op(op, None, st, self.ws if lane == 0 else self.lane_ws[lane])
                if i in needed:
                    self._mark(i).record(st)
            for j in joins:
                self._mark(j).wait(cur)
        if self.net.loss == "softmax_xent":
            self.loss_fwd_bwd(trace, stream)

    def _forward_op(self, op, trace, stream, ws):
        x = self.act[op.src]
        if op.name in self.merged:
            y, w, b = self.m_act[op.name], self.mWlp[op.name], self.mb[op.name]
            if trace: trace("conv_bias_relu_fwd", op, stream=stream, x=x, w=w, b=b, y=y)
            ops.conv2d_fwd_bias_relu(x, w, b, (1, 1), op.pads, y=y, ws=ws, stream=stream)
            if trace: trace("conv_bias_relu_fwd:end", op, stream=stream, y=y)
            return
        y = self._slice(self.act, op)
        if isinstance(op, Conv) and not op.relu:
            # a classifier's logits: the bias is added inside the cross-entropy kernel
            if trace: trace("conv_fwd", op, stream=stream, x=x, w=self.Wlp[op.name], y=y)
            ops.conv2d_fwd(x, self.Wlp[op.name], (op.sh, op.sw), op.pads, y=y, ws=ws, stream=stream)
            if trace: trace("conv_fwd:end", op, stream=stream, y=y)
        elif isinstance(op, Conv) and op.name in self.conv_pool:
            pool = self.conv_pool[op.name]
            py, am = self._slice(self.act, pool), self.argmax[pool.name]
            if trace: trace("conv_bias_relu_maxpool_fwd", op, stream=stream, x=x, w=self.Wlp[op.name],
                            b=self.b[op.name], y=y, py=py, argmax=am)
            ops.conv2d_fwd_bias_relu_maxpool(x, self.Wlp[op.name], self.b[op.name], (op.sh, op.sw), op.pads,
                                             (pool.kh, pool.kw), (pool.sh, pool.sw), pool.pads, y=y, py=py,
                                             taps=am, ws=ws, stream=stream)
            if trace: trace("conv_bias_relu_maxpool_fwd:end", op, stream=stream, y=y, py=py, argmax=am)
        elif isinstance(op, Pool) and op.name in self.pool_in_conv:
            return                           # produced with its convolution
        elif isinstance(op, Conv):
            if trace: trace("conv_bias_relu_fwd", op, stream=stream, x=x, w=self.Wlp[op.name],
                            b=self.b[op.name], y=y)
            ops.conv2d_fwd_bias_relu(x, self.Wlp[op.name], self.b[op.name], (op.sh, op.sw), op.pads, y=y,
                                     ws=ws, stream=stream)
            if trace: trace("conv_bias_relu_fwd:end", op, stream=stream, y=y)
        else:
            if trace: trace("maxpool_fwd", op, stream=stream, x=x, y=y, argmax=self.argmax[op.name])
            ops.maxpool_fwd(x, (op.kh, op.kw), (op.sh, op.sw), op.pads, y=y, argmax=self.argmax[op.name],
                            stream=stream)
            if trace: trace("maxpool_fwd:end", op, stream=stream, y=y, argmax=self.argmax[op.name])

    def loss_fwd_bwd(self, trace=None, stream=None):
        """Mean softmax cross-entropy of the logits (the logits layer's bias added here) and its
        gradient (softmax - onehot) / N, written as the upstream gradient of the logits."""
        net = self.net
        fc = next(op for op in net.ops if isinstance(op, Conv) and op.dst == net.output)
        logits, bias = self.act[net.output], self.b[fc.name]
        if trace: trace("softmax_xent", fc, stream=stream, logits=logits, bias=bias, labels=self.labels)
        ops.softmax_xent(logits, self.labels, 1.0 / logits.shape[0], bias=bias, loss=self.loss_rows,
                         dlogits=self.g, stream=stream)
        if trace: trace("softmax_xent:end", fc, stream=stream, loss=self.loss_rows, dlogits=self.g)

    def loss_value(self) -> float:
        """The last step's batch-mean cross-entropy (host copy; synchronises)."""
        return float(self.loss_rows.double().mean())

    def _relu_backward(self, op, dy, trace, stream, defer, jobs, grouped, lws):
        """The ReLU (or bias-only) backward of convolution ``op``'s output gradient ``dy``, unless a
        fused kernel forms it (a pool's or a consumer's input gradient); returns the gradient
        before the ReLU, the one its filter and input gradients read."""
        net = self.net
        if not op.relu:
            dpre = dy                        # bias only: the gradient passes through
            if trace: trace("bias_bwd", op, stream=stream, dy=dy)
            if defer:
                ws = self._bias_ws(("bias", op.name), ops.bias_relu_bwd_workspace_bytes(dy))
                jobs.append((ops.bias_relu_bwd(None, dy, dpre=dpre, ws=ws, stream=stream, defer=True)[1],
                             self.db[op.name]))
            else:
                ops.bias_relu_bwd(None, dy, dpre=dpre, dbias=self.db[op.name], ws=lws, stream=stream)
            if trace: trace("bias_bwd:end", op, stream=stream, dpre=dpre, db=self.db[op.name])
        elif op.name in self.relu_fused:
            dpre = dy                        # written by the fused pool / input-gradient backward
        elif op.name in self.relu_groups:
            dpre = dy
            c0, width, run = self.relu_groups[op.name]
            if id(run) not in grouped:       # the group's last convolution in forward order
                grouped.add(id(run))
                yg, dyg = self.act[op.dst][..., c0:c0 + width], self.grad[op.dst][..., c0:c0 + width]
                dbg = self.grads[self._layout[run[0].name][2]:self._layout[run[0].name][2] + width]
                if trace: trace("bias_relu_bwd", op, stream=stream, y=yg, dy=dyg)
                if defer:
                    ws = self._bias_ws(("group", op.dst, c0), ops.bias_relu_bwd_workspace_bytes(yg))
                    jobs.append((ops.bias_relu_bwd(yg, dyg, dpre=dyg, ws=ws, stream=stream, defer=True)[1],
                                 dbg))
                else:
                    ops.bias_relu_bwd(yg, dyg, dpre=dyg, dbias=dbg, ws=lws, stream=stream)
                if trace: trace("bias_relu_bwd:end", op, stream=stream, dpre=dyg, db=dbg)
        else:
            y = self._slice(self.act, op)
            dpre = self._slice({op.dst: self.dpre_out}, op) if op.dst == net.output else dy
            if trace: trace("bias_relu_bwd", op, stream=stream, y=y, dy=dy)
            if defer:
                ws = self._bias_ws(("relu", op.name), ops.bias_relu_bwd_workspace_bytes(y))
                jobs.append((ops.bias_relu_bwd(y, dy, dpre=dpre, ws=ws, stream=stream, defer=True)[1],
                             self.db[op.name]))
            else:
                ops.bias_relu_bwd(y, dy, dpre=dpre, dbias=self.db[op.name], ws=lws, stream=stream)
            if trace: trace("bias_relu_bwd:end", op, stream=stream, dpre=dpre, db=self.db[op.name])
        return dpre

    def _input_grad_relu_last(self, op, dpre, w, beta, trace, stream, defer, jobs, grouped, lws):
        """The input gradient of convolution ``op`` as the last of its input's readers, fused with
        the ReLU backward of the group of convolutions that produced the whole input."""
        t, (c0, width, run) = self.relu_last[op.name]
        y, dx = self.act[t], self.grad[t]
        bo = self._layout[run[0].name][2]
        dbg = self.grads[bo:bo + width]
        grouped.add(id(run))
        if trace: trace("conv_bwd_input_relu_bwd", op, stream=stream, dy=dpre, w=w, y=y, dpre=dx, beta=beta)
        if defer:
            ws = self._bias_ws(("last", op.name), ops.conv2d_workspace_bytes(
                3, y, op.cout, op.kh, op.kw, (op.sh, op.sw), op.pads))
            jobs.append((ops.conv2d_bwd_input_relu_bwd(dpre, w, y, dx, (op.sh, op.sw), op.pads, ws=ws, stream=stream,
                                                       defer=True, beta=beta)[1], dbg))
        else:
            ops.conv2d_bwd_input_relu_bwd(dpre, w, y, dx, (op.sh, op.sw), op.pads, dbias=dbg, ws=lws,
                                          stream=stream, beta=beta)
        if trace: trace("conv_bwd_input_relu_bwd:end", op, stream=stream, dpre=dx, db=dbg)

    def backward(self, trace=None, stream=None, side=None, lanes=True):
        """Gradients of every variable.  With ``side`` (a second stream), the filter gradient
        of each convolution that also has an input gradient runs there, concurrently with that
        input gradient and everything after it on ``stream``: the two only read the same
        tensors, and the side stream joins back before this returns (the dataflow executor runs
        independent kernels on several GPU streams, Section 5)."""
        cur = stream if stream is not None else torch.cuda.current_stream()
        # (traced steps form each bias gradient at once, so that the tracer can check it)
        defer = trace is None and self.defer_bias
        jobs = []                                # deferred bias gradients: (partials, dbias)
        state = (set(), set(), jobs, defer)      # gradients written so far, ReLU groups done
        if trace is not None or not lanes or not self.lane_streams or torch.cuda.is_current_stream_capturing():
            for op in reversed(self.ops):
                self._backward_node(op, trace, stream, side, self.ws, state)
        else:
            plan, joins = self.bwd_plan
            needed = {j for _, _, waits in plan for j in waits} | set(joins)
            if "start" in needed:
                self._mark(("b", "start")).record(cur)
            for i, (op, lane, waits) in enumerate(plan):
                st = cur if lane == 0 else self.lane_streams[lane + 1]
                for j in waits:
                    self._mark(("b", j)).wait(st)
                self._backward_node(op, None, st, side, self.ws if lane == 0 else self.lane_ws[lane + 1], state)
                if i in needed:
                    self._mark(("b", i)).record(st)
            for j in joins:
                self._mark(("b", j)).wait(cur)
        if jobs:
            ops.bias_grad_finish(jobs, stream=stream)
        if side is not None:
            ops.stream_wait(cur, side)

    def _backward_node(self, op, trace, stream, side, ws, state):
        """One op's gradients: its ReLU (or bias) backward, its filter gradient (on ``side`` when
        given and the op has an input gradient too) and its input gradient, on ``stream`` with
        workspace ``ws``."""
        net = self.net
        written, grouped, jobs, defer = state
        cur = stream if stream is not None else torch.cuda.current_stream()
        dy = self._slice(self.grad, op) if op.name not in self.merged else None
        src_grad = op.src != "x" or net.input_grad
        beta = 1.0 if op.src in written else 0.0
        if op.name in self.merged:
            # each member's ReLU backward (most are fused into other kernels), then the merged
            # filter and input gradients over the members' adjacent gradient channels
            for m in self.merged[op.name]["members"]:
                self._relu_backward(m, self._slice(self.grad, m), trace, stream, defer, jobs, grouped, ws)
            dpre, x = self.m_grad[op.name], self.act[op.src]
            on_side = side is not None and src_grad
            if on_side:
                ops.stream_wait(side, cur)
            fs = side if on_side else stream
            dw = self.mdW[op.name]
            if trace: trace("conv_bwd_filter", op, stream=fs, x=x, dy=dpre)
            ops.conv2d_bwd_filter(x, dpre, (1, 1), (1, 1), op.pads, dw=dw,
                                  ws=self.ws_side if on_side else ws, stream=fs)
            if trace: trace("conv_bwd_filter:end", op, stream=fs, dw=dw)
            if src_grad and op.name in self.relu_last:
                self._input_grad_relu_last(op, dpre, self.mWlp[op.name], beta, trace, stream, defer, jobs,
                                           grouped, ws)
                written.add(op.src)
            elif src_grad:
                dx, w = self.grad[op.src], self.mWlp[op.name]
                if trace: trace("conv_bwd_input", op, stream=stream, dy=dpre, w=w, dx=dx, beta=beta)
                ops.conv2d_bwd_input(dpre, w, dx, (1, 1), op.pads, beta=beta, ws=ws, stream=stream)
                if trace: trace("conv_bwd_input:end", op, stream=stream, dx=dx)
                written.add(op.src)
            return
        if isinstance(op, Conv):
            dpre = self._relu_backward(op, dy, trace, stream, defer, jobs, grouped, ws)
            x = self.act[op.src]
            # a filter gradient with no input gradient beside it (the first layer) stays
            # on the main stream, where it is next on the critical path
            on_side = side is not None and src_grad
            if on_side:
                ops.stream_wait(side, cur)
            fs = side if on_side else stream
            if trace: trace("conv_bwd_filter", op, stream=fs, x=x, dy=dpre)
            ops.conv2d_bwd_filter(x, dpre, (op.kh, op.kw), (op.sh, op.sw), op.pads, dw=self.dW[op.name],
                                  ws=self.ws_side if on_side else ws, stream=fs)
            if trace: trace("conv_bwd_filter:end", op, stream=fs, dw=self.dW[op.name])
            if src_grad and op.name in self.bwi_relu:
                prod = self.bwi_relu[op.name]
                dx, y = self.grad[op.src], self.act[op.src]
                if trace: trace("conv_bwd_input_relu_bwd", op, stream=stream, dy=dpre, w=self.Wlp[op.name],
                                y=y)
                if defer:
                    ws = self._bias_ws(("bwi", op.name), ops.conv2d_workspace_bytes(
                        3, y, op.cout, op.kh, op.kw, (op.sh, op.sw), op.pads))
                    jobs.append((ops.conv2d_bwd_input_relu_bwd(dpre, self.Wlp[op.name], y, dx, (op.sh, op.sw),
                                                               op.pads, ws=ws, stream=stream, defer=True)[1],
                                 self.db[prod.name]))
                else:
                    ops.conv2d_bwd_input_relu_bwd(dpre, self.Wlp[op.name], y, dx, (op.sh, op.sw), op.pads,
                                                  dbias=self.db[prod.name], ws=ws, stream=stream)
                if trace: trace("conv_bwd_input_relu_bwd:end", op, stream=stream, dpre=dx, db=self.db[prod.name])
            elif src_grad and op.name in self.relu_last:
                self._input_grad_relu_last(op, dpre, self.Wlp[op.name], beta, trace, stream, defer, jobs,
                                           grouped, ws)
            elif src_grad:
                dx = self.grad[op.src]
                if trace: trace("conv_bwd_input", op, stream=stream, dy=dpre, w=self.Wlp[op.name], dx=dx,
                                beta=beta)
                ops.conv2d_bwd_input(dpre, self.Wlp[op.name], dx, (op.sh, op.sw), op.pads, beta=beta,
                                     ws=ws, stream=stream)
                if trace: trace("conv_bwd_input:end", op, stream=stream, dx=dx)
        elif op.name in self.pool_relu:
            conv = self.pool_relu[op.name]
            y, dpre, am = self.act[op.src], self.grad[op.src], self.argmax[op.name]
            py = self._slice(self.act, op)
            if trace: trace("maxpool_relu_bwd", op, stream=stream, dy=dy, argmax=am, y=y, py=py, dpre=dpre,
                            beta=beta)
            # (the pool's output gives the ReLU mask where the gradient is not accumulated)
            if defer:
                ws = self._bias_ws(("pool", op.name), ops.bias_relu_bwd_workspace_bytes(dpre))
                jobs.append((ops.maxpool_bwd_relu_bwd(dy, am, y, dpre, (op.kh, op.kw), (op.sh, op.sw), op.pads,
                                                      beta=beta, ws=ws, stream=stream, py=py, defer=True)[1],
                             self.db[conv.name]))
            else:
                ops.maxpool_bwd_relu_bwd(dy, am, y, dpre, (op.kh, op.kw), (op.sh, op.sw), op.pads, beta=beta,
                                         dbias=self.db[conv.name], ws=ws, stream=stream, py=py)
            if trace: trace("maxpool_relu_bwd:end", op, stream=stream, dpre=dpre, db=self.db[conv.name])
        elif src_grad and op.name in self.relu_last:
            # the last reader of a concat: its pool gradient added, then the concat's ReLU backward
            t, (c0, width, run) = self.relu_last[op.name]
            y, dpre, am = self.act[t], self.grad[t], self.argmax[op.name]
            bo = self._layout[run[0].name][2]
            dbg = self.grads[bo:bo + width]
            grouped.add(id(run))
            py = self._slice(self.act, op)
            if trace: trace("maxpool_relu_bwd", op, stream=stream, dy=dy, argmax=am, y=y, py=py, dpre=dpre,
                            beta=beta)
            if defer:
                ws = self._bias_ws(("last", op.name), ops.bias_relu_bwd_workspace_bytes(dpre))
                jobs.append((ops.maxpool_bwd_relu_bwd(dy, am, y, dpre, (op.kh, op.kw), (op.sh, op.sw), op.pads,
                                                      beta=beta, ws=ws, stream=stream, py=py, defer=True)[1],
                             dbg))
            else:
                ops.maxpool_bwd_relu_bwd(dy, am, y, dpre, (op.kh, op.kw), (op.sh, op.sw), op.pads, beta=beta,
                                         dbias=dbg, ws=ws, stream=stream, py=py)
            if trace: trace("maxpool_relu_bwd:end", op, stream=stream, dpre=dpre, db=dbg)
        else:
            if src_grad:
                dx = self.grad[op.src]
                am = self.argmax[op.name]
                if trace: trace("maxpool_bwd", op, stream=stream, dy=dy, argmax=am, dx=dx, beta=beta)
                ops.maxpool_bwd(dy, am, dx, (op.kh, op.kw), (op.sh, op.sw), op.pads, beta=beta,
                                stream=stream)
                if trace: trace("maxpool_bwd:end", op, stream=stream, dx=dx)
        if src_grad:
            written.add(op.src)

    def update(self, trace=None, stream=None):
        a = self.opt_args
        self.t += 1
        if self.optimizer == "sgd":
            if trace: trace("apply_sgd", None, stream=stream, var=self.params, grad=self.grads)
            ops.apply_sgd(self.params, self.grads, self.lr, shadow=self.shadow, stream=stream)
            if trace: trace("apply_sgd:end", None, stream=stream, var=self.params)
        elif self.optimizer == "momentum":
            if trace: trace("apply_momentum", None, stream=stream, var=self.params, grad=self.grads)
            ops.apply_momentum(self.params, self.slots[0], self.grads, self.lr, a["momentum"], a["nesterov"],
                               shadow=self.shadow, stream=stream)
            if trace: trace("apply_momentum:end", None, stream=stream, var=self.params)
        else:
            if trace: trace("apply_adam", None, stream=stream, var=self.params, grad=self.grads)
            ops.apply_adam(self.params, self.slots[0], self.slots[1], self.grads, self.lr, a["beta1"], a["beta2"],
                           a["epsilon"], self.t, shadow=self.shadow, stream=stream)
            if trace: trace("apply_adam:end", None, stream=stream, var=self.params)

    def step(self, trace=None, stream=None, concurrent=True):
        """One training step on ``stream``; unless ``concurrent`` is false, the forward pass's
        independent branches run side by side on the lane streams and the filter gradients
        overlap the rest of the backward pass on a second stream.  ``trace(event, op,
        stream=s, **tensors)`` is called before and after every op (``event`` ending in
        ``:end``), with the stream the op runs on (None: the current stream)."""
        self.forward(trace, stream, lanes=concurrent)
        self.backward(trace, stream, side=self.side if concurrent else None)
        self.update(trace, stream)

    def record_step(self, stream=None, concurrent=True) -> "ops.Program":
        """Runs one step (as ``step``) while recording its library calls into a program, which
        ``run_program`` issues again for every later step from C++ (the cached step subgraph of
        Sections 3.2 and 3.3).  The update is recorded too, except Adam's, whose bias correction
        depends on the step count: ``run_program`` then runs it after the recorded calls."""
        prog = ops.Program()
        prog.with_update = self.optimizer != "adam"
        with prog.recording():
            self.forward(None, stream, lanes=concurrent)
            self.backward(None, stream, side=self.side if concurrent else None)
            if prog.with_update:
                self.update(None, stream)
        if not prog.with_update:
            self.update(None, stream)
        # (the recorded stream joins name this replica's marks by pointer: the program keeps them)
        prog.marks = dict(self.marks)
        return prog

    def run_program(self, prog, stream=None):
        """One training step from a program made by ``record_step`` (on the streams it was
        recorded on; ``stream`` only places an update that was not recorded)."""
        prog.run()
        if prog.with_update:
            self.t += 1
        else:
            self.update(None, stream)

    # ------------------------------------------------------------------ state
    def snapshot(self):
        """Copies of the variables (master and shadow), the optimizer slots and the step count,
        for restore-and-rerun checks."""
        return (self.params.clone(), None if self.shadow is None else self.shadow.clone(),
                [t.clone() for t in self.slots], self.t)

    def restore(self, snap):
        self.params.copy_(snap[0])
        if self.shadow is not None:
            self.shadow.copy_(snap[1])
        for t, v in zip(self.slots, snap[2]):
            t.copy_(v)
        self.t = snap[3]
