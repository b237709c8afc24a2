"""Device memory plumbing: weights, KV pool and workspace as torch tensors on
one GPU, bound to an hxf instance.  PyTorch only allocates memory and supplies
the stream; every computation runs in libhxf.so."""
import numpy as np
import torch

from . import hxf


def _dev_u16(bits, device):
    a = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(a).to(device)


def _dev_packed(bits, device):
    """Upload a row-major bf16 [N, K] weight and repack it on the GPU into the
    library's MFMA tile layout (the row-major copy is dropped)."""
    n, k = bits.shape
    src = _dev_u16(bits, device)
    out = torch.empty(hxf.packed_weight_bytes(n, k) // 2, dtype=torch.int16, device=device)
    hxf.op_pack_weight(src.data_ptr(), n, k, out.data_ptr(), torch.cuda.current_stream(device).cuda_stream)
    return out


class DeviceModel:
    """Weights of one decoder in HBM (bf16 bit patterns in int16 tensors).

    ``layer_fn(l)`` returns the host bf16 bits of layer l as a dict with keys
    wq, wk, wv, wo, w_gate, w_up, w_down; ``embed``, ``lm_head`` and ``norm``
    are host bf16 bits.  Wq, Wk and Wv are stacked row-wise into one QKV matrix.
    Projection matrices and the LM head are held packed (hxf_op_pack_weight).
    ``norm`` is one bf16 gain [d] used by every RMSNorm, or a dict with one gain
    per norm: attn [L, d], ffn [L, d], final [d].
    """

    def __init__(self, shape, layer_fn, embed, lm_head, norm, device="cuda"):
        self.shape = shape
        self.device = device
        self.embed = _dev_u16(embed, device)
        self.lm_head = _dev_packed(lm_head, device)
        L = shape.n_layers
        if isinstance(norm, dict):
            self.norm = _dev_u16(norm["final"], device)
            self.attn_norm = [_dev_u16(norm["attn"][l], device) for l in range(L)]
            self.ffn_norm = [_dev_u16(norm["ffn"][l], device) for l in range(L)]
        else:
            self.norm = _dev_u16(norm, device)
            self.attn_norm = [self.norm] * L
            self.ffn_norm = [self.norm] * L
        self.layers = []
        for l in range(shape.n_layers):
            w = layer_fn(l)
            qkv = np.concatenate([w["wq"], w["wk"], w["wv"]], axis=0)
            self.layers.append({
                "wqkv": _dev_packed(qkv, device), "wo": _dev_packed(w["wo"], device),
                "w_gate": _dev_packed(w["w_gate"], device), "w_up": _dev_packed(w["w_up"], device),
                "w_down": _dev_packed(w["w_down"], device),
            })
        torch.cuda.current_stream(device).synchronize()

    def layer_ptrs(self):
        return [{"attn_norm": a.data_ptr(), "ffn_norm": f.data_ptr(), **{k: t.data_ptr() for k, t in L.items()}}
                for a, f, L in zip(self.attn_norm, self.ffn_norm, self.layers)]


class Engine:
    """An hxf instance bound to a DeviceModel, a KV pool and a workspace."""

    def __init__(self, model, max_context, n_blocks, max_seqs, chunk_tokens, cost_ps, iter_ps,
                 policy=hxf.POLICY_PQ, clock=hxf.CLOCK_VIRTUAL, stream=None):
        self.model = model
        self.mcfg = hxf.model_cfg(model.shape, max_context)
        self.scfg = hxf.sched_cfg(n_blocks, max_seqs, chunk_tokens, cost_ps, iter_ps, policy, clock, hxf.EXEC_HIP)
        self.inst = hxf.Instance(self.mcfg, self.scfg)
        kvb = hxf.kv_pool_bytes(self.mcfg, n_blocks)
        wsb = hxf.workspace_bytes(self.mcfg, self.scfg)
        self.kv_pool = torch.empty(kvb, dtype=torch.uint8, device=model.device)
        self.workspace = torch.empty(wsb, dtype=torch.uint8, device=model.device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(model.device)
        self.inst.bind(model.embed.data_ptr(), model.norm.data_ptr(), model.lm_head.data_ptr(), model.layer_ptrs(),
                       self.kv_pool.data_ptr(), kvb, self.workspace.data_ptr(), wsb, self.stream.cuda_stream)

    def layer_kv(self, layer):
        """(K pool, V pool) views of one layer: [Hkv, n_blocks, dh/8, 16, 8] and [Hkv, n_blocks, dh, 16] (int16 bits)."""
        sh = self.model.shape
        nb = self.scfg.n_blocks
        per = nb * sh.n_kv_heads * 16 * sh.head_dim
        flat = self.kv_pool.view(torch.int16)
        k = flat[(2 * layer) * per:(2 * layer + 1) * per].view(sh.n_kv_heads, nb, sh.head_dim // 8, 16, 8)
        v = flat[(2 * layer + 1) * per:(2 * layer + 2) * per].view(sh.n_kv_heads, nb, sh.head_dim, 16)
        return k, v
