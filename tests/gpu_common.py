"""Helpers for the GPU parity tests: run the HIP path through the C ABI,
bring its outputs back in the oracle's canonical layouts, compare."""
from __future__ import annotations

import numpy as np

import paper_2608_27875_amd as hyq
from oracle import hyq_oracle as orc

TOL_MAX = 2e-3
TOL_MEAN = 2e-4


def to_dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def shape_of(cfg) -> hyq.Shape:
    return hyq.Shape(B=cfg["B"], Hq=cfg["Hq"], Hkv=cfg["Hkv"], L=cfg["L"], D=cfg.get("D", 128),
                     window=cfg["W"], budget_ppm=cfg["budget_ppm"], bits_kv=cfg["bits"],
                     kv_format=cfg.get("fmt", hyq.FMT_INT))


def fmt_name(shape) -> str:
    """Oracle format name of a Shape or a decode cache struct."""
    return {hyq.FMT_FP8: "fp8", hyq.FMT_FP4: "fp4", hyq.FMT_FP4Q6: "fp4q6"}.get(shape.kv_format,
                                                                               "int")


def run_gpu(shape: hyq.Shape, d, out_dtype=0, keep_out_on_gpu=False, tensors=None):
    """One pass select -> quantize -> attention through the C ABI."""
    import torch
    if tensors is None:
        tensors = tuple(to_dev(d[n]) for n in ("Q", "K", "V"))
    Q, K, V = tensors
    bufs = hyq.alloc_buffers(shape, Q.device, out_dtype)
    z = bufs["sizes"]
    scores = torch.empty(z["scores_bytes"] // 4, dtype=torch.float32, device=Q.device) \
        if z["k"] > 0 else None
    hyq.hyq_select_vertical(shape, Q, K, bufs["idx"], scores, bufs["ws"])
    hyq.hyq_quantize(shape, Q, K, V, bufs["idx"], bufs["q_codes"], bufs["q_scale"],
                     bufs["k_codes"], bufs["k_scale"], bufs["v_codes"], bufs["v_scale"],
                     bufs["kq_pos"])
    hyq.hyq_attn_prefill(shape, Q, K, V, bufs["idx"], bufs["q_codes"], bufs["q_scale"],
                         bufs["k_codes"], bufs["k_scale"], bufs["v_codes"], bufs["v_scale"],
                         bufs["kq_pos"], 1.0 / np.sqrt(shape.D), bufs["out"], out_dtype)
    torch.cuda.synchronize()
    g = {n: bufs[n].cpu().numpy() for n in
         ("idx", "q_codes", "q_scale", "k_codes", "k_scale", "v_codes", "v_scale", "kq_pos")}
    g["scores"] = None if scores is None else scores.cpu().numpy()
    g["sizes"] = z
    if keep_out_on_gpu:
        g["out_dev"] = bufs["out"]
    else:
        o = bufs["out"]
        g["out"] = (o.float() if out_dtype else o).cpu().numpy()
    return g


def unpack_codes4(raw: np.ndarray, fmt: int) -> np.ndarray:
    """Packed 4-bit codes -> one code per element: two's-complement int4
    values, or E2M1 codes 0..15 for FP4."""
    if fmt in (hyq.FMT_FP4, hyq.FMT_FP4Q6):
        out = np.empty(raw.shape[:-1] + (raw.shape[-1] * 2,), dtype=np.uint8)
        out[..., 0::2] = raw & 0xF
        out[..., 1::2] = raw >> 4
        return out
    return _nibbles(raw)


def _nibbles(raw: np.ndarray) -> np.ndarray:
    """uint8 [..., n] of packed two's-complement nibbles -> int8 [..., 2n]
    (element 2i = low nibble of byte i)."""
    lo = (raw & 0xF).astype(np.int16)
    hi = (raw >> 4).astype(np.int16)
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(raw.shape[:-1] + (raw.shape[-1] * 2,), dtype=np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


def canonical(shape: hyq.Shape, g: dict) -> dict:
    """GPU buffers -> the oracle's layouts (codes [B,H,nQ,D] int8), checking
    that padding slots hold the documented values."""
    z = g["sizes"]
    B, Hq, Hkv, L, D = shape.B, shape.Hq, shape.Hkv, shape.L, shape.D
    nQ, nb = z["nQ"], z["n_kvblk"]
    slots = nb * 64
    kq = g["kq_pos"].reshape(B, Hkv, slots)
    assert np.all(kq[..., nQ:] == hyq.KQ_POS_PAD)
    ctype = np.int8 if shape.kv_format == hyq.FMT_INT else np.uint8
    out = dict(kq_pos=kq[..., :nQ],
               q_codes=g["q_codes"].view(ctype).reshape(B, Hq, L, D),
               q_scale=g["q_scale"].reshape(B, Hq, z["n_qblk"]),
               k_scale=g["k_scale"].reshape(B, Hkv, nb),
               v_scale=g["v_scale"].reshape(B, Hkv, nb))
    if shape.bits_kv == 8:
        kc = g["k_codes"].view(ctype).reshape(B, Hkv, slots, D)
        vc = g["v_codes"].view(ctype).reshape(B, Hkv, nb, D, 64)
    else:
        kc = unpack_codes4(g["k_codes"].view(np.uint8).reshape(B, Hkv, slots, D // 2),
                           shape.kv_format)
        vc = unpack_codes4(g["v_codes"].view(np.uint8).reshape(B, Hkv, nb, D, 32), shape.kv_format)
    vc = vc.transpose(0, 1, 2, 4, 3).reshape(B, Hkv, slots, D)
    assert np.all(kc[:, :, nQ:] == 0) and np.all(vc[:, :, nQ:] == 0)
    out["k_codes"] = kc[:, :, :nQ]
    out["v_codes"] = vc[:, :, :nQ]
    return out


def check_select_quant(shape: hyq.Shape, d: dict, g: dict):
    """Bit-exact comparison of selection and quantization with the oracle;
    returns (idx, qz) of the oracle for the attention comparison."""
    idx, S = orc.select_vertical(d["Q"], d["K"], shape.Hkv, shape.window, shape.budget_ppm)
    z = g["sizes"]
    assert idx.shape == (shape.B, shape.Hkv, z["k"])
    np.testing.assert_array_equal(g["idx"].reshape(idx.shape), idx)
    if z["k"] > 0:
        gs = g["scores"].reshape(S.shape)
        np.testing.assert_array_equal(gs.view(np.uint32), S.view(np.uint32))
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, shape.window, shape.bits_kv,
                      fmt=fmt_name(shape) if shape.bits_kv != 16 else "int")
    if shape.bits_kv != 16:
        c = canonical(shape, g)
        for key in ("kq_pos", "q_codes", "k_codes", "v_codes"):
            np.testing.assert_array_equal(c[key], qz[key], err_msg=key)
        for key in ("q_scale", "k_scale", "v_scale"):
            np.testing.assert_array_equal(c[key].view(np.uint32), qz[key].view(np.uint32),
                                          err_msg=key)
    return idx, qz


def sample_rows(L: int, W: int, n: int, seed: int) -> np.ndarray:
    """n query rows: always 0, P-1, P, L-1 (the ends of the prefix and the
    window), the rest drawn without replacement."""
    P = max(0, L - W)
    must = sorted({0, max(0, P - 1), min(P, L - 1), L - 1})
    rng = np.random.default_rng(seed)
    pool = np.setdiff1d(np.arange(L), must)
    extra = rng.choice(pool, size=min(len(pool), max(0, n - len(must))), replace=False)
    return np.array(sorted(set(must) | set(extra.tolist())), dtype=np.int64)


def scaled_error(O_gpu: np.ndarray, O_ref: np.ndarray):
    """Max error of each row divided by max(1, max |O_ref| of the row): the
    bound for inputs whose outputs are far above 1, where f16 weights limit
    the accuracy relative to the output's own size."""
    err = np.abs(O_gpu.astype(np.float64) - O_ref.astype(np.float64))
    scale = np.maximum(1.0, np.abs(O_ref.astype(np.float64)).max(axis=-1, keepdims=True))
    return float((err / scale).max())


def attention_error(O_gpu: np.ndarray, O_ref: np.ndarray):
    err = np.abs(O_gpu.astype(np.float64) - O_ref.astype(np.float64))
    return float(err.max()), float(err.mean())
