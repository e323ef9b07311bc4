"""Layer-chain builder: turns a list of layer specs plus their float
parameters into a device-resident ifq_stack and runs it with ifq_run_stack.

This is the "convert once, then deploy" step of IFQ-Net (Sec. 3): weights are
packed and thresholds folded once, on the host, by the library's own C++
entry points, then uploaded; a forward pass is one ifq_run_stack call that
launches every layer on one stream without host synchronisation.

Layer specs are duck-typed. A conv spec has name, src, dst, h, w, cin, cout,
k, stride, pad, in_bits, out_bits and join (None, ("identity", slot) or
("conv", slot, down_layer_name)); a pool spec has name, src, dst, h, w, c, k,
stride, mode ("valid" / "same") and bits. Slot "x" is the stack input, "y"
the output. Parameters of a conv are a dict with w (OIHW +-1 int8), alpha,
bias, mean, var, gamma, bn_beta (per output channel), eps, beta_in, q_thr.
"""
import ctypes

import numpy as np

from . import _ffi, api
from ._ffi import (Layer, Stack, IFQ_LAYER_CONV, IFQ_LAYER_POOL, IFQ_LAYER_CONV_POOL,
                   IFQ_LAYER_CONV_FP4, IFQ_LAYER_CONV_POOL_FP4,
                   IFQ_LAYOUT_I8_NHWC, IFQ_LAYOUT_U2_NHWC_PACKED,
                   IFQ_LAYOUT_I32_NHWC, IFQ_LAYOUT_U2_BLOCK64, IFQ_JOIN_NONE, IFQ_JOIN_IDENTITY,
                   IFQ_JOIN_CONV, IFQ_JOIN_CONV_FUSED, IFQ_POOL_VALID, IFQ_POOL_SAME)


def _is_conv(L):
    return hasattr(L, "cin")


_POOL_MODE = {"valid": IFQ_POOL_VALID, "same": IFQ_POOL_SAME}


def _pool_hw(h, w, P):
    """Output size of pool spec P over h x w (as ifq_maxpool_codes)."""
    if P.mode == "valid":
        return (h - P.k) // P.stride + 1, (w - P.k) // P.stride + 1
    return -(-h // P.stride), -(-w // P.stride)


def conv_ops(L, batch):
    """Dense int-ops of a conv layer: 2 * N*Ho*Wo * Cout * kh*kw*Cin."""
    ho = (L.h + 2 * L.pad - L.k) // L.stride + 1
    wo = (L.w + 2 * L.pad - L.k) // L.stride + 1
    return 2 * batch * ho * wo * L.cout * L.k * L.k * L.cin


class DeviceStack:
    """A stack of quantized substructures resident on one GPU.

    code_layout: layout of the 2-bit code tensors: "i8" (one byte per
    code), "u2" (NHWC, four codes per byte, for channel counts that are
    multiples of 16) or "b64" (channel blocks of 64 for channel counts that
    are multiples of 64, else as "u2"). Other tensors use one byte per code;
    int32 sums stay int32. The stack input and output are NHWC codes on the
    host side either way (upload_input / download_output convert).
    fuse_down: with "b64", compute each 1x1 downsample inside the conv join
    that consumes it (IFQ_JOIN_CONV_FUSED); self.fused maps the join's layer
    name to the downsample's, whose layer and output tensor are then absent.
    fuse_pool: a conv whose codes only the following max-pool reads runs as
    one IFQ_LAYER_CONV_POOL layer where a fused kernel covers the pair
    (ifq_conv_pool_kernel_name). True fuses the pools whose windows tile the
    conv output (valid, k == stride), where the fused kernel keeps its usual
    tile count; "all" also the others, which the fused kernels run with one
    image per tile (slower than a separate pool at small batch: too few
    workgroups for the chip). fp4: the convs an fp4 kernel covers (the
    windowed kernel's 2-bit threshold layers) run on it (IFQ_LAYER_CONV_FP4,
    the same codes); self.fp4_layers names them. self.fused_pool maps
    the conv's name to the pool's, whose layer and the conv's output tensor
    are then absent.
    """

    def __init__(self, layers, params, batch, code_layout="i8",
                 device="cuda", fuse_down=False, fuse_pool=False, fp4=False):
        import torch
        if code_layout not in ("i8", "u2", "b64"):
            raise ValueError("code_layout must be 'i8', 'u2' or 'b64'")
        all_layers = list(layers)
        by_name = {L.name: (i, L) for i, L in enumerate(all_layers)}
        # fuse_down (BLOCK64 codes): a 1x1 downsample whose int32 sums only a
        # conv join reads runs inside that join's kernel (IFQ_JOIN_CONV_FUSED);
        # its layer and its output tensor disappear from the stack
        self.fused = {}
        if fuse_down and code_layout == "b64":
            for L in all_layers:
                if not (_is_conv(L) and L.join is not None and L.join[0] == "conv"):
                    continue
                D = by_name[L.join[2]][1]
                readers = [M for M in all_layers if M.name != L.name and
                           (M.src == D.dst or (_is_conv(M) and M.join is not None
                                               and M.join[1] == D.dst))]
                if (not readers and D.k == 1 and D.pad == 0 and D.in_bits == 2 and
                        D.cin % 64 == 0 and L.cout % 64 == 0 and L.k == 3 and
                        L.pad == 1 and L.cin % 64 == 0 and L.out_bits == 2):
                    self.fused[L.name] = D.name
        skip = set(self.fused.values())
        self._all_layers = all_layers
        self.layers = [L for L in all_layers if L.name not in skip]
        self.batch = int(batch)
        self.fp4_layers = []
        self.fused_pool = {}
        if fuse_pool:
            self.fused_pool = self._pool_fusions(code_layout, fuse_pool)
            drop = set(self.fused_pool.values())
            self.layers = [L for L in self.layers if L.name not in drop]
        pool_of = {c: by_name[p][1] for c, p in self.fused_pool.items()}
        src_index = [by_name[L.name][0] for L in self.layers]
        self.device = torch.device(device)
        self._keep = []
        slots = {"x": 0, "y": 1}
        layout_of = {}

        def sid(name):
            if name not in slots:
                slots[name] = len(slots)
            return slots[name]

        def code_layout_for(bits, channels):
            if code_layout == "b64" and bits == 2 and channels % 64 == 0:
                return IFQ_LAYOUT_U2_BLOCK64
            if code_layout in ("u2", "b64") and bits == 2 and channels % 16 == 0:
                return IFQ_LAYOUT_U2_NHWC_PACKED
            return IFQ_LAYOUT_I8_NHWC

        L0 = self.layers[0]
        c0 = L0.cin if _is_conv(L0) else L0.c
        b0 = L0.in_bits if _is_conv(L0) else L0.bits
        layout_of["x"] = code_layout_for(b0, c0)
        self.input_shape = (self.batch, L0.h, L0.w, c0)
        self.input_bits = b0
        self.input_layout = layout_of["x"]

        self.tensor_info = {"x": (self.input_shape, layout_of["x"], b0)}
        # slot -> (the layer specs' name of the tensor it holds last, the spec
        # layer that computed it: a fused pool's name for a fused conv + pool)
        self.slot_origin = {"x": ("x", None)}
        alias = {}

        def cur(name):
            return alias.get(name, name)
        arr = (Layer * len(self.layers))()
        self.ops = 0
        for i, L in enumerate(self.layers):
            rec = arr[i]
            # slot names: a fused conv + pool that would read and write the
            # same slot (slots ping-pong along the chain) writes a slot of its
            # own, which stands for that name until the name is written again
            src_name = cur(L.src)
            if L.name in pool_of:
                dst_name = pool_of[L.name].dst
                if cur(dst_name) == src_name:
                    alias[dst_name] = "%s@%s" % (dst_name, L.name)
                else:
                    alias.pop(dst_name, None)
                dst_name, orig_dst, writer = cur(dst_name), dst_name, pool_of[L.name].name
            else:
                alias.pop(L.dst, None)
                dst_name, orig_dst, writer = L.dst, L.dst, L.name
            rec.src = sid(src_name)
            rec.dst = sid(dst_name)
            rec.join_src = -1
            in_layout = layout_of[src_name]
            if _is_conv(L):
                p = params[src_index[i]]
                rec.kind = IFQ_LAYER_CONV
                if L.out_bits == 0:
                    out_layout = IFQ_LAYOUT_I32_NHWC
                else:
                    out_layout = code_layout_for(L.out_bits, L.cout)
                d = api.conv_desc(self.batch, L.h, L.w, L.cin, L.cout, L.k,
                                  L.stride, L.pad, L.in_bits, L.out_bits,
                                  in_layout, out_layout)
                rec.conv = d
                if L.name in pool_of:
                    Pl = pool_of[L.name]
                    rec.kind = IFQ_LAYER_CONV_POOL
                    ho, wo = api.ifq_conv_output_dims(d)
                    rec.pool = api.pool_desc(self.batch, ho, wo, L.cout, Pl.k, Pl.stride,
                                             _POOL_MODE[Pl.mode], L.out_bits, out_layout)
                blob = api.ifq_pack_weights(d, p["w"])
                wdev = torch.from_numpy(blob).to(self.device)
                self._keep.append(wdev)
                rec.w_packed = wdev.data_ptr()
                if L.out_bits != 0 and L.join is None:
                    thr = api.ifq_fold_thresholds(
                        L.cout, L.in_bits, L.out_bits, L.k * L.k * L.cin,
                        p["alpha"], p["beta_in"], p["q_thr"], bias=p.get("bias"),
                        mean=p["mean"], var=p["var"], gamma=p["gamma"],
                        bn_beta=p["bn_beta"], eps=p["eps"])
                    tdev = torch.from_numpy(thr).to(self.device)
                    self._keep.append(tdev)
                    rec.thr = tdev.data_ptr()
                if L.join is not None:
                    if L.join[0] == "identity":
                        # the shortcut is the block input: codes with the
                        # input's step beta_in
                        table = api.ifq_fold_join_table(
                            p, p["beta_in"], L.in_bits, L.k * L.k * L.cin,
                            L.out_bits, p["q_thr"])
                        tdev = torch.from_numpy(table).to(self.device)
                        self._keep.append(tdev)
                        rec.join = api.make_join(IFQ_JOIN_IDENTITY,
                                                 layout_of[cur(L.join[1])], None, None,
                                                 p["q_thr"], table=tdev)
                    elif L.name in self.fused:
                        D = by_name[self.fused[L.name]][1]
                        pd = params[by_name[D.name][0]]
                        coef = api.ifq_fold_join(IFQ_JOIN_CONV, p, pd["beta_in"],
                                                 down=pd)
                        cdev = torch.from_numpy(coef).to(self.device)
                        dd = api.conv_desc(self.batch, D.h, D.w, D.cin, D.cout, D.k,
                                           D.stride, D.pad, D.in_bits, 0,
                                           layout_of[cur(D.src)], IFQ_LAYOUT_I32_NHWC)
                        ddev = torch.from_numpy(api.ifq_pack_weights(dd, pd["w"])).to(
                            self.device)
                        self._keep += [cdev, ddev]
                        rec.join = api.make_join(IFQ_JOIN_CONV_FUSED, layout_of[cur(D.src)],
                                                 None, cdev, p["q_thr"], down_w=ddev,
                                                 down=dd)
                        self.ops += conv_ops(D, self.batch)
                    else:
                        pd = params[by_name[L.join[2]][0]]
                        coef = api.ifq_fold_join(IFQ_JOIN_CONV, p, pd["beta_in"],
                                                 down=pd)
                        cdev = torch.from_numpy(coef).to(self.device)
                        self._keep.append(cdev)
                        rec.join = api.make_join(IFQ_JOIN_CONV, layout_of[cur(L.join[1])],
                                                 None, cdev, p["q_thr"])
                    rec.join_src = (sid(cur(by_name[self.fused[L.name]][1].src))
                                    if L.name in self.fused else sid(cur(L.join[1])))
                if (fp4 and rec.kind == IFQ_LAYER_CONV and
                        (L.join is None or L.join[0] == "identity" or L.name in self.fused)
                        and api.ifq_conv_fp4_kernel_name(d, rec.join if L.join else None)):
                    # the same layer on the fp4 path: its own weight blob (and
                    # the fused downsample's)
                    rec.kind = IFQ_LAYER_CONV_FP4
                    self.fp4_layers.append(L.name)
                    w4 = torch.from_numpy(api.ifq_pack_weights_fp4(d, p["w"])).to(self.device)
                    self._keep.append(w4)
                    rec.w_packed = w4.data_ptr()
                    if L.name in self.fused:
                        D = by_name[self.fused[L.name]][1]
                        pd = params[by_name[D.name][0]]
                        d4 = torch.from_numpy(api.ifq_pack_weights_fp4(
                            rec.join.down, pd["w"])).to(self.device)
                        self._keep.append(d4)
                        rec.join.down_w = d4.data_ptr()
                elif (fp4 and rec.kind == IFQ_LAYER_CONV_POOL and
                      api.ifq_conv_pool_fp4_kernel_name(d, rec.pool)):
                    rec.kind = IFQ_LAYER_CONV_POOL_FP4
                    self.fp4_layers.append(L.name)
                    w4 = torch.from_numpy(api.ifq_pack_weights_fp4(d, p["w"])).to(self.device)
                    self._keep.append(w4)
                    rec.w_packed = w4.data_ptr()
                self.ops += conv_ops(L, self.batch)
                ho, wo = api.ifq_conv_output_dims(d)
                out_shape = (self.batch, ho, wo, L.cout)
                out_bits = L.out_bits
                if L.name in pool_of:
                    out_shape = (self.batch,) + _pool_hw(ho, wo, pool_of[L.name]) + (L.cout,)
            else:
                rec.kind = IFQ_LAYER_POOL
                mode = {"valid": IFQ_POOL_VALID, "same": IFQ_POOL_SAME}[L.mode]
                out_layout = in_layout
                rec.pool = api.pool_desc(self.batch, L.h, L.w, L.c, L.k,
                                         L.stride, mode, L.bits, in_layout)
                if mode == IFQ_POOL_VALID:
                    ho, wo = (L.h - L.k) // L.stride + 1, (L.w - L.k) // L.stride + 1
                else:
                    ho, wo = -(-L.h // L.stride), -(-L.w // L.stride)
                out_shape = (self.batch, ho, wo, L.c)
                out_bits = L.bits
            layout_of[dst_name] = out_layout
            self.tensor_info[dst_name] = (out_shape, out_layout, out_bits)
            self.slot_origin[dst_name] = (orig_dst, writer)
            if dst_name == "y":
                self.output_shape = out_shape
                self.output_layout = out_layout
                self.output_bits = out_bits
        self._layers = arr
        self.n_slots = len(slots)
        self.slots = dict(slots)
        self.stack = Stack(len(self.layers), self.n_slots,
                           ctypes.cast(arr, ctypes.POINTER(Layer)), None)
        nbytes = api.ifq_stack_workspace_bytes(self.stack)
        if nbytes == 0 and self.n_slots > 2:
            raise api.IfqError(-1, "ifq_stack_workspace_bytes",
                               api.ifq_last_error())
        # zero-filled once: the K-split arrival counters at its start must
        # be zero before the first run (every run leaves them zero)
        self.ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8,
                              device=self.device)

    def _pool_fusions(self, code_layout, fuse=True):
        """conv name -> pool name for every conv whose codes only the
        following max-pool reads and whose pair a fused kernel covers (layouts
        as the stack would give them)."""
        layout_of = {}

        def code_layout_for(bits, channels):
            if code_layout == "b64" and bits == 2 and channels % 64 == 0:
                return IFQ_LAYOUT_U2_BLOCK64
            if code_layout in ("u2", "b64") and bits == 2 and channels % 16 == 0:
                return IFQ_LAYOUT_U2_NHWC_PACKED
            return IFQ_LAYOUT_I8_NHWC

        L0 = self.layers[0]
        layout_of[L0.src] = code_layout_for(L0.in_bits if _is_conv(L0) else L0.bits,
                                            L0.cin if _is_conv(L0) else L0.c)
        out = {}
        for i, L in enumerate(self.layers):
            if not _is_conv(L):
                layout_of[L.dst] = layout_of[L.src]
                continue
            out_layout = (IFQ_LAYOUT_I32_NHWC if L.out_bits == 0
                          else code_layout_for(L.out_bits, L.cout))
            layout_of[L.dst] = out_layout
            nxt = self.layers[i + 1] if i + 1 < len(self.layers) else None
            if (nxt is None or _is_conv(nxt) or nxt.src != L.dst or L.join is not None
                    or L.out_bits == 0 or L.dst == "y"):
                continue
            ho0 = (L.h + 2 * L.pad - L.k) // L.stride + 1
            wo0 = (L.w + 2 * L.pad - L.k) // L.stride + 1
            rows = (nxt.mode == "valid" and nxt.k == nxt.stride and ho0 % nxt.k == 0
                    and wo0 % nxt.k == 0)
            if not rows and fuse != "all":
                continue
            # anything reading the conv's tensor before its slot is written
            # again (slots are reused along the chain)
            read_later = False
            for M in self.layers[i + 2:]:
                if M.src == L.dst or (_is_conv(M) and M.join is not None
                                      and M.join[1] == L.dst):
                    read_later = True
                    break
                if M.dst == L.dst:
                    break
            if read_later:
                continue
            d = api.conv_desc(self.batch, L.h, L.w, L.cin, L.cout, L.k, L.stride, L.pad,
                              L.in_bits, L.out_bits, layout_of[L.src], out_layout)
            ho, wo = api.ifq_conv_output_dims(d)
            pd = api.pool_desc(self.batch, ho, wo, L.cout, nxt.k, nxt.stride,
                               _POOL_MODE[nxt.mode], L.out_bits, out_layout)
            if api.ifq_conv_pool_kernel_name(d, pd):
                out[L.name] = nxt.name
        return out

    # -- buffers ---------------------------------------------------------------
    def _bytes(self, shape, layout):
        n, h, w, c = shape
        return api.ifq_tensor_bytes(n, h, w, c, layout)

    def alloc_input(self):
        import torch
        return torch.empty(self._bytes(self.input_shape, self.input_layout),
                           dtype=torch.uint8, device=self.device)

    def alloc_output(self):
        import torch
        return torch.empty(self._bytes(self.output_shape, self.output_layout),
                           dtype=torch.uint8, device=self.device)

    def upload_input(self, codes, out=None):
        """NHWC uint8 codes (host) -> device input in the stack's layout."""
        import torch
        codes = np.ascontiguousarray(codes, dtype=np.uint8)
        assert codes.shape == self.input_shape, (codes.shape, self.input_shape)
        if out is None:
            out = self.alloc_input()
        src = torch.from_numpy(codes.reshape(-1)).to(self.device)
        if self.input_layout != IFQ_LAYOUT_I8_NHWC:
            n, h, w, c = self.input_shape
            api.ifq_convert_codes(n, h, w, c, IFQ_LAYOUT_I8_NHWC,
                                  self.input_layout, src, out)
        else:
            out.copy_(src)
        return out

    def download_output(self, y):
        """Device output -> host NHWC array (uint8 codes or int32 sums)."""
        import torch
        n, h, w, c = self.output_shape
        if self.output_layout == IFQ_LAYOUT_I32_NHWC:
            return y.view(torch.int32).cpu().numpy().reshape(n, h, w, c)
        if self.output_layout != IFQ_LAYOUT_I8_NHWC:
            full = torch.empty(n * h * w * c, dtype=torch.uint8, device=self.device)
            api.ifq_convert_codes(n, h, w, c, self.output_layout,
                                  IFQ_LAYOUT_I8_NHWC, y, full)
            return full.cpu().numpy().reshape(n, h, w, c)
        return y.cpu().numpy().reshape(n, h, w, c)

    def read_slot(self, name):
        """Host copy of a work slot's last tensor (after a run has finished):
        NHWC uint8 codes or int32 sums; 2-bit codes are returned as stored
        (uint8 [n][h][w][c/4] for "u2", [n][c/64][h][w][16] for "b64")."""
        import torch
        (n, h, w, c), layout, _ = self.tensor_info[name]
        off, _ = api.ifq_stack_slot_info(self.stack, self.slots[name])
        nb = self._bytes((n, h, w, c), layout)
        raw = self.ws[off:off + nb]
        if layout == IFQ_LAYOUT_I32_NHWC:
            return raw.view(torch.int32).cpu().numpy().reshape(n, h, w, c)
        if layout == IFQ_LAYOUT_U2_NHWC_PACKED:
            return raw.cpu().numpy().reshape(n, h, w, c // 4)
        if layout == IFQ_LAYOUT_U2_BLOCK64:
            return raw.cpu().numpy().reshape(n, c // 64, h, w, 16)
        return raw.cpu().numpy().reshape(n, h, w, c)

    def layer_kernel_names(self):
        """Kernel each layer launches (conv variants by name, pools as
        maxpool_codes)."""
        out = []
        for i, L in enumerate(self.layers):
            lay = self._layers[i]
            if lay.kind == IFQ_LAYER_CONV_POOL:
                out.append(api.ifq_conv_pool_kernel_name(lay.conv, lay.pool))
            elif lay.kind == IFQ_LAYER_CONV_FP4:
                join = lay.join if lay.join.kind != IFQ_JOIN_NONE else None
                out.append(api.ifq_conv_fp4_kernel_name(lay.conv, join))
            elif lay.kind == IFQ_LAYER_CONV_POOL_FP4:
                out.append(api.ifq_conv_pool_fp4_kernel_name(lay.conv, lay.pool))
            elif _is_conv(L):
                join = lay.join if lay.join.kind != IFQ_JOIN_NONE else None
                out.append(api.ifq_conv_kernel_name(lay.conv, join))
            else:
                out.append("maxpool_codes")
        return out

    def layer_ops(self):
        """Dense int-ops of every layer (0 for pools; a conv with a fused
        downsample counts both convs)."""
        names = {L.name: L for L in self._all_layers}
        out = []
        for L in self.layers:
            ops = conv_ops(L, self.batch) if _is_conv(L) else 0
            if L.name in self.fused:
                ops += conv_ops(names[self.fused[L.name]], self.batch)
            out.append(ops)
        return out

    # -- execution -------------------------------------------------------------
    def _slot_ptr(self, k, x, y):
        if k == 0:
            return x.data_ptr()
        if k == 1:
            return y.data_ptr()
        off, _ = api.ifq_stack_slot_info(self.stack, k)
        return self.ws.data_ptr() + off

    def layer_launcher(self, i, x, y, stream=None):
        """A callable that launches layer i alone on the stack's buffers
        (asynchronous), exactly as ifq_run_stack launches it: same
        descriptor, weights, thresholds, join and slots. Valid once a full
        run has filled the layer's input slots. The arguments are marshalled
        once, so repeated calls cost one C call each."""
        rec = self._layers[i]
        lib = _ffi.load()
        vp = ctypes.c_void_p
        src = vp(self._slot_ptr(rec.src, x, y))
        dst = vp(self._slot_ptr(rec.dst, x, y))
        st = api._stream(stream)
        if rec.kind == IFQ_LAYER_CONV:
            desc = rec.conv
            join = None
            if rec.join.kind != 0:
                join = _ffi.Join.from_buffer_copy(rec.join)
                join.shortcut = self._slot_ptr(rec.join_src, x, y)
            # the stack workspace: its conv region (offset 0) is what
            # ifq_run_stack hands a K-split layer
            args = (ctypes.byref(desc), src, vp(rec.w_packed), vp(rec.thr),
                    None if join is None else ctypes.byref(join), dst, None,
                    vp(self.ws.data_ptr()), self.ws.numel(), st)
            fn = lib.ifq_conv_forward
            what = "ifq_conv_forward"
        elif rec.kind == IFQ_LAYER_CONV_FP4:
            desc = rec.conv
            join = None
            if rec.join.kind != 0:
                join = _ffi.Join.from_buffer_copy(rec.join)
                join.shortcut = self._slot_ptr(rec.join_src, x, y)
            args = (ctypes.byref(desc), src, vp(rec.w_packed), vp(rec.thr),
                    None if join is None else ctypes.byref(join), dst, st)
            fn = lib.ifq_conv_forward_fp4
            what = "ifq_conv_forward_fp4"
        elif rec.kind in (IFQ_LAYER_CONV_POOL, IFQ_LAYER_CONV_POOL_FP4):
            desc = (rec.conv, rec.pool)
            join = None
            args = (ctypes.byref(rec.conv), ctypes.byref(rec.pool), src, vp(rec.w_packed),
                    vp(rec.thr), dst, st)
            f4 = rec.kind == IFQ_LAYER_CONV_POOL_FP4
            fn = lib.ifq_conv_pool_forward_fp4 if f4 else lib.ifq_conv_pool_forward
            what = "ifq_conv_pool_forward_fp4" if f4 else "ifq_conv_pool_forward"
        else:
            desc = rec.pool
            args = (ctypes.byref(desc), src, dst, st)
            fn = lib.ifq_maxpool_codes
            what = "ifq_maxpool_codes"

        def launch():
            api._check(fn(*args), what)
        launch.keep = (desc, join if rec.kind != IFQ_LAYER_POOL else None)
        return launch

    def run_static(self, x, y, stream=None):
        """One forward pass on the library's static workspace
        (ifq_run_stack_static) instead of self.ws."""
        self.stack.events = None
        api.ifq_run_stack_static(self.stack, x, y, stream)

    def run(self, x, y, stream=None, events=None):
        """One forward pass (asynchronous on stream). events: optional ctypes
        array of n_layers + 1 hipEvent_t handles for per-layer timing."""
        self.stack.events = (None if events is None
                             else ctypes.cast(events, ctypes.c_void_p).value)
        api.ifq_run_stack(self.stack, x, y, self.ws, stream)
