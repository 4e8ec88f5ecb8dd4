"""Seeded synthetic refresh-step workloads.

This module only lays out sequences and draws random numbers; it holds none
of the method's arithmetic, and both the HIP path and the CPU oracle consume
the exact bytes it produces.

The paper's datasets are not used.  Inputs stand in for its workloads:
single-image prompts (the K = 1 benchmarks of Sec. 4.1), multi-image prompts,
a 16k-token multi-image context (the latency setting of Sec. 4.3) and long
multi-page documents.  The distributions are:

  * K and Q ~ N(0, 1) elementwise at every position, so a plain logit at scale
    1/sqrt(d) is ~N(0, 1);
  * V_t = rho_t * u_t with u_t uniform on the sphere of the H_kv*d concatenated
    heads and rho_t ~ LogNormal(0, 0.5), so the value-norm proxy is rho_t;
  * sinks: keys 3*sqrt(d)*b_kv along a per-KV-head unit vector b, every span
    query gets +2*b, and the sink's rho is multiplied by 0.05 (high attention,
    small value norm);
  * relevant images: keys sqrt(0.7)*z + sqrt(0.3)*sqrt(d)*w_kv and span
    queries sqrt(0.7)*z' + sqrt(0.3)*sqrt(d)*w_kv with w orthogonal to b
    (query-key cosine ~0.3);
  * fresh rows for the refresh follow the isotropic staleness model of the
    Monte Carlo estimator (App. D.1) with kappa = 0.5:
    K*_t = K_t + xi, xi ~ N(0, kappa^2 ||K_t||^2 / (H_kv d) I), same for V*;
    fresh queries Q*_t ~ N(0, 1) (drawn in float32);
  * the text rows a refresh also recomputes (every non-visual position) get
    fresh K/V and queries drawn the same way, on streams of their own;
  * the residual-error diagnostic draws M standard normal direction samples
    per visual token over the concatenated H_kv*d value dims (M = 5 in App.
    D.1), in the cache dtype.

Sequence layout: [changed prefix][for each image: separator, visual tokens]
[span].  Caches are token-major [N_ctx, H_kv, d].  bf16 arrays are returned as
uint16 bit patterns (round-to-nearest-even from float32).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

# random stream ids
(_S_Q, _S_K, _S_VDIR, _S_VNORM, _S_SINK, _S_REL, _S_XI, _S_QSTAR, _S_XI_TEXT, _S_QSTAR_TEXT,
 _S_ISO) = range(11)
_GLOBAL_LAYER = 65535  # stream for draws shared by all layers


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float -> bf16 bit patterns (uint16), round to nearest even via float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> 16) & np.uint32(1)
    u = u + np.uint32(0x7FFF)   # finite values never wrap
    u += lsb
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32, exactly."""
    return (np.asarray(bits).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Workload:
    cfg_id: int
    name: str
    dtype: str                      # "f32" or "bf16"
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_q: int
    q_pos0: int
    n_ctx: int
    img_pos: np.ndarray             # int32 [K]
    img_off: np.ndarray             # int32 [K+1]
    n_sinks: int
    n_relevant: int
    budgets: Dict[str, int]         # label -> k
    seed: int = 0
    lognormal_sigma: float = 0.5
    kappa: float = 0.5
    rel_cos: float = 0.3            # query-key cosine of relevant images

    @property
    def n_images(self) -> int:
        return len(self.img_pos)

    @property
    def n_vis(self) -> int:
        return int(self.img_off[-1])

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def vis_positions(self) -> np.ndarray:
        """Sequence position of every visual token (layout bookkeeping)."""
        return np.concatenate([np.arange(p, p + (self.img_off[j + 1] - self.img_off[j]))
                               for j, p in enumerate(self.img_pos)]).astype(np.int64)

    # -- random streams ---------------------------------------------------
    def _rng(self, layer: int, stream: int) -> np.random.Generator:
        return np.random.default_rng([self.seed, self.cfg_id, layer, stream])

    def _cast(self, x: np.ndarray) -> np.ndarray:
        if self.dtype == "f32":
            return np.ascontiguousarray(x, dtype=np.float32)
        return bf16_bits(x)

    def shared(self) -> dict:
        """Draws shared by every layer: sink ids, relevant image ids, b, w."""
        d, hkv, nv = self.head_dim, self.n_kv_heads, self.n_vis
        rs = self._rng(_GLOBAL_LAYER, _S_SINK)
        sinks = np.sort(rs.choice(nv, size=self.n_sinks, replace=False)) if self.n_sinks else \
            np.zeros(0, np.int64)
        b = rs.standard_normal((hkv, d))
        b /= np.linalg.norm(b, axis=1, keepdims=True)
        rr = self._rng(_GLOBAL_LAYER, _S_REL)
        rel = np.sort(rr.choice(self.n_images, size=self.n_relevant, replace=False)) \
            if self.n_relevant else np.zeros(0, np.int64)
        w = rr.standard_normal((hkv, d))
        w -= np.sum(w * b, axis=1, keepdims=True) * b
        w /= np.linalg.norm(w, axis=1, keepdims=True)
        return {"sinks": sinks, "relevant": rel, "b": b, "w": w}

    def text_positions(self) -> np.ndarray:
        """Positions outside the images (prefix, separators, span), ascending."""
        keep = np.ones(self.n_ctx, dtype=bool)
        keep[self.vis_positions()] = False
        return np.flatnonzero(keep).astype(np.int64)

    def layer(self, layer: int, fresh: bool = True, text: bool = False) -> dict:
        """All tensors of one layer, already cast to the cache dtype.

        q [n_q, H_q, d]; k, v [N_ctx, H_kv, d]; with fresh=True also
        q_star [N_vis, H_q, d], k_star, v_star [N_vis, H_kv, d] (fresh rows in
        visual-index order); with text=True also q_text_star, k_text_star,
        v_text_star for the rows of text_positions(), in that order.
        """
        d, hq, hkv, nq, nctx = self.head_dim, self.n_q_heads, self.n_kv_heads, self.n_q, \
            self.n_ctx
        sh = self.shared()
        P_vis = self.vis_positions()
        g = self.group

        q = self._rng(layer, _S_Q).standard_normal((nq, hq, d))
        k = self._rng(layer, _S_K).standard_normal((nctx, hkv, d))
        u = self._rng(layer, _S_VDIR).standard_normal((nctx, hkv * d))
        u /= np.linalg.norm(u, axis=1, keepdims=True)
        rho = self._rng(layer, _S_VNORM).lognormal(0.0, self.lognormal_sigma, size=nctx)

        head_kv = np.arange(hq) // g
        if self.n_relevant:
            zq = q
            rc = self.rel_cos
            q = np.sqrt(1 - rc) * zq + np.sqrt(rc) * np.sqrt(d) * sh["w"][head_kv][None, :, :]
            for j in sh["relevant"]:
                lo = int(self.img_pos[j])
                hi = lo + int(self.img_off[j + 1] - self.img_off[j])
                k[lo:hi] = np.sqrt(1 - rc) * k[lo:hi] + np.sqrt(rc) * np.sqrt(d) * sh["w"][None]
        if self.n_sinks:
            q = q + 2.0 * sh["b"][head_kv][None, :, :]
            sp = P_vis[sh["sinks"]]
            k[sp] = 3.0 * np.sqrt(d) * sh["b"][None]
            rho[sp] *= 0.05
        v = (rho[:, None] * u).reshape(nctx, hkv, d)

        out = {"q": self._cast(q), "k": self._cast(k), "v": self._cast(v)}
        if fresh:
            rx = self._rng(layer, _S_XI)
            kv_vis = k[P_vis]
            vv_vis = v[P_vis]
            sd_k = self.kappa * np.linalg.norm(kv_vis.reshape(len(P_vis), -1), axis=1) / \
                np.sqrt(hkv * d)
            sd_v = self.kappa * np.linalg.norm(vv_vis.reshape(len(P_vis), -1), axis=1) / \
                np.sqrt(hkv * d)
            k_star = kv_vis + sd_k[:, None, None] * rx.standard_normal(kv_vis.shape)
            v_star = vv_vis + sd_v[:, None, None] * rx.standard_normal(vv_vis.shape)
            out["k_star"] = self._cast(k_star)
            out["v_star"] = self._cast(v_star)
            out["q_star"] = self._cast(self._rng(layer, _S_QSTAR).standard_normal(
                (len(P_vis), hq, d), dtype=np.float32))
        if text:
            T = self.text_positions()
            rx = self._rng(layer, _S_XI_TEXT)
            kt, vt = k[T], v[T]
            sd_k = self.kappa * np.linalg.norm(kt.reshape(len(T), -1), axis=1) / np.sqrt(hkv * d)
            sd_v = self.kappa * np.linalg.norm(vt.reshape(len(T), -1), axis=1) / np.sqrt(hkv * d)
            out["k_text_star"] = self._cast(kt + sd_k[:, None, None] * rx.standard_normal(kt.shape))
            out["v_text_star"] = self._cast(vt + sd_v[:, None, None] * rx.standard_normal(vt.shape))
            out["q_text_star"] = self._cast(self._rng(layer, _S_QSTAR_TEXT).standard_normal(
                (len(T), hq, d), dtype=np.float32))
        return out


def iso_directions(w: "Workload", layer: int, n_samples: int) -> np.ndarray:
    """Standard normal draws z [n_samples, N_vis, H_kv, d] in the cache dtype."""
    z = w._rng(layer, _S_ISO).standard_normal((n_samples, w.n_vis, w.n_kv_heads, w.head_dim),
                                                dtype=np.float32)
    return w._cast(z)


def _layout(prefix: int, n_img: int, per_img: int, sep: int, n_q: int):
    img_pos, img_off = [], [0]
    cur = prefix
    for _ in range(n_img):
        cur += sep
        img_pos.append(cur)
        cur += per_img
        img_off.append(img_off[-1] + per_img)
    return (np.array(img_pos, np.int32), np.array(img_off, np.int32), cur, cur + n_q)


def config(cfg_id: int, seed: int = 0, n_layers: Optional[int] = None) -> Workload:
    """The five refresh-step workloads (1-based ids).

    1: one layer, one image of 576 tokens after a 64-token changed prefix,
       32 span tokens, 8 heads MHA, d 64, fp32, 5 sinks, 10% budget.
    2: one layer, one image of 1,024 tokens after a 256-token prefix, 64 span
       tokens, GQA 28/4, d 128, bf16, 2% sinks, 10% budget.
    3: 28 layers, 4 images x 1,296 tokens after a 128-token prefix, 96 span
       tokens aligned with 1 relevant image, bf16, 5/10/20% budgets.
    4: one layer, 16 images x 1,024 tokens (16,384), each after a 16-token
       separator, 512-token prefix, 128 span tokens, 3 relevant images,
       bf16, 10% budget.
    5: 28 layers, 64 pages x 1,024 tokens (65,536) after a 1,024-token prefix,
       256 span tokens, 1% sinks, 4 relevant pages, bf16, 10% budget.
    """
    if cfg_id == 1:
        ip, io, q0, nctx = _layout(64, 1, 576, 0, 32)
        w = Workload(1, "1 image x 576 vis + 64 prefix, 32 queries, MHA 8x64, fp32", "f32", 1,
                     8, 8, 64, 32, q0, nctx, ip, io, 5, 0, {"10%": 57, "10%-stated": 58})
    elif cfg_id == 2:
        ip, io, q0, nctx = _layout(256, 1, 1024, 0, 64)
        w = Workload(2, "1 image x 1024 vis + 256 prefix, 64 queries, GQA 28/4x128, bf16", "bf16",
                     1, 28, 4, 128, 64, q0, nctx, ip, io, 20, 0, {"10%": 102})
    elif cfg_id == 3:
        ip, io, q0, nctx = _layout(128, 4, 1296, 0, 96)
        w = Workload(3, "28 layers, 4 images x 1296 vis + 128 prefix, 96 queries, GQA 28/4x128, "
                     "bf16", "bf16", 28, 28, 4, 128, 96, q0, nctx, ip, io, 0, 1,
                     {"5%": 259, "10%": 518, "20%": 1036})
    elif cfg_id == 4:
        ip, io, q0, nctx = _layout(512, 16, 1024, 16, 128)
        w = Workload(4, "16 images x 1024 vis (16384) + 16-token separators + 512 prefix, "
                     "128 queries, GQA 28/4x128, bf16", "bf16", 1, 28, 4, 128, 128, q0, nctx, ip,
                     io, 0, 3, {"10%": 1638})
    elif cfg_id == 5:
        ip, io, q0, nctx = _layout(1024, 64, 1024, 0, 256)
        w = Workload(5, "28 layers, 64 pages x 1024 vis (65536) + 1024 prefix, 256 queries, "
                     "GQA 28/4x128, bf16", "bf16", 28, 28, 4, 128, 256, q0, nctx, ip, io, 655, 4,
                     {"10%": 6553, "10%-stated": 6554})
    else:
        raise ValueError(f"unknown workload {cfg_id}")
    w.seed = seed
    if n_layers is not None:
        w.n_layers = n_layers
    return w


def custom(n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int, n_q: int,
           prefix: int, images: List[int], sep: int, dtype: str, n_sinks: int = 0,
           n_relevant: int = 0, seed: int = 0, cfg_id: int = 100) -> Workload:
    """A small workload of arbitrary shape (for tests: ragged tails, odd sizes)."""
    img_pos, img_off, cur = [], [0], prefix
    for n in images:
        cur += sep
        img_pos.append(cur)
        cur += n
        img_off.append(img_off[-1] + n)
    return Workload(cfg_id, "custom", dtype, n_layers, n_q_heads, n_kv_heads, head_dim, n_q, cur,
                    cur + n_q, np.array(img_pos, np.int32), np.array(img_off, np.int32), n_sinks,
                    n_relevant, {}, seed)
