"""Seeded synthetic inputs for the subspace-network (SSN) stage-boundary codec.

This module only draws random numbers and builds input tensors: bases U, the
fixed token-embedding table E, token ids, activations X, gradients G, weight
matrices W, and the coordinate/noise draws Z0 and eta that tests combine into
structured activations.  It holds none of the codec's arithmetic (no
projection, no gather-and-subtract, no reconstruction), so that the oracle and
the HIP path can both consume the same inputs without sharing any computation.

Two backends produce the same distributions:

* host (numpy) -- exact, used for the small and mid configurations and every
  structured construction the tests need;
* device (torch generator on a GPU) -- used for the full-size workloads, where
  host generation of a 1 GiB embedding table would dominate a benchmark run.

Shapes and distributions follow the paper's Pluralis-8B stage boundary
(section 4.1 "Pipeline-Parallel Communication with Reparameterized SSNs" and
the model card of section 5.2), scaled to the five workloads listed in
``CONFIGS``.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Sequence

import numpy as np

# Independent random streams per input kind, so that e.g. changing the noise
# level never changes the basis or the ids.
STREAM = {"U": 0, "E": 1, "ids": 2, "Z0": 3, "noise": 4, "X": 5, "G": 6, "W": 7,
          "perm": 8, "sel": 9, "uZipf": 10, "theta": 11, "drift": 12, "P": 13,
          "progress": 14}


def rng(seed: int, stream: str) -> np.random.Generator:
    """Counter-free numpy generator for one (seed, input kind) pair."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), STREAM[stream]])))


# --------------------------------------------------------------------------
# bf16 storage: the host keeps bf16 tensors as uint16 bit patterns.
# --------------------------------------------------------------------------
def to_bf16_bits(x) -> np.ndarray:
    """Round float values to bfloat16 (round-to-nearest-even), as uint16 bits."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def store(x, dtype: str) -> np.ndarray:
    """Round a float array to the storage dtype ('f32' -> float32, 'bf16' -> uint16 bits)."""
    if dtype == "f32":
        return np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    if dtype == "bf16":
        return to_bf16_bits(x)
    raise ValueError(f"unknown dtype {dtype!r}")


# --------------------------------------------------------------------------
# Bases U (d x k).  The paper does not say how U_k is built (it cites the SSN
# work for that); any orthonormal basis serves.  Three families are provided.
# --------------------------------------------------------------------------
def gaussian_orthonormal_basis(d: int, k: int, seed: int) -> np.ndarray:
    """QR of a seeded N(0,1) d x k matrix, signs fixed so diag(R) > 0 (float64)."""
    a = rng(seed, "U").standard_normal((d, k))
    q, r = np.linalg.qr(a)
    s = np.sign(np.diag(r))
    s[s == 0] = 1.0
    return np.ascontiguousarray(q * s)


def hadamard_basis(d: int, k: int, seed: int = 0) -> np.ndarray:
    """k distinct columns of the Sylvester-Hadamard matrix H_d / sqrt(d).

    With d = 4**m every entry is +-2**-m, exactly representable in bf16 and
    fp32, so the stored basis is exactly orthonormal.
    """
    if d < 1 or d & (d - 1):
        raise ValueError("d must be a power of two")
    h = np.array([[1.0]])
    while h.shape[0] < d:
        h = np.block([[h, h], [h, -h]])
    cols = np.sort(rng(seed, "sel").choice(d, size=k, replace=False))
    return np.ascontiguousarray(h[:, cols] / np.sqrt(d))


def selection_basis(d: int, k: int, seed: int = 0) -> np.ndarray:
    """k distinct columns of the identity I_d (exact in every dtype)."""
    cols = rng(seed, "sel").choice(d, size=k, replace=False)
    u = np.zeros((d, k))
    u[cols, np.arange(k)] = 1.0
    return u


# --------------------------------------------------------------------------
# Token ids.
# --------------------------------------------------------------------------
def zipf_cdf(V: int, s: float) -> np.ndarray:
    """CDF of the Zipf law truncated to ranks 1..V: p(r) proportional to r**-s."""
    w = np.arange(1, V + 1, dtype=np.float64) ** (-float(s))
    c = np.cumsum(w)
    return c / c[-1]


def token_ids(N: int, V: int, seed: int, dist: str = "uniform", zipf_s: float = 1.1) -> np.ndarray:
    """int32 ids in [0, V).  'zipf': ranks by inverse CDF, scattered over the
    vocabulary by a seeded permutation (frequent tokens are not the low ids)."""
    if dist == "uniform":
        return rng(seed, "ids").integers(0, V, size=N, dtype=np.int64).astype(np.int32)
    if dist == "zipf":
        u = rng(seed, "uZipf").random(N)
        rank = np.searchsorted(zipf_cdf(V, zipf_s), u, side="right")
        rank = np.minimum(rank, V - 1)
        perm = rng(seed, "perm").permutation(V)
        return perm[rank].astype(np.int32)
    raise ValueError(f"unknown id distribution {dist!r}")


# --------------------------------------------------------------------------
# Workload configurations.
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class CodecConfig:
    name: str
    B: int
    S: int
    d: int
    k: int
    V: int
    dtype: str            # 'f32' or 'bf16'
    seed: int
    structured: bool      # X = E[ids] + Z0 U^T + eta  (else X ~ N(0,1))
    noise_std: float = 0.0
    emb_std: float = 0.02
    ids_dist: str = "uniform"
    zipf_s: float = 1.1

    @property
    def N(self) -> int:
        return self.B * self.S


@dataclasses.dataclass(frozen=True)
class WeightsConfig:
    name: str
    d: int
    k: int
    layers: int
    shapes: Sequence[tuple]   # per layer: (rows=d, cols=n) of each subspace-constrained matrix
    dtype: str
    seed: int
    w_std: float = 0.02


TINY = CodecConfig("tiny_f32", B=4, S=128, d=256, k=8, V=1024, dtype="f32", seed=1001,
                   structured=True, noise_std=1e-3)
MID = CodecConfig("mid_bf16", B=8, S=1024, d=2048, k=32, V=32768, dtype="bf16", seed=1002,
                  structured=True, noise_std=1e-2)
STAGE8B = CodecConfig("stage8b_bf16", B=16, S=2048, d=4096, k=64, V=131072, dtype="bf16",
                      seed=1003, structured=False)
WEIGHTS = WeightsConfig("weights_stage4", d=4096, k=64, layers=4,
                        shapes=((4096, 4096), (4096, 14336)), dtype="bf16", seed=1004)


def sweep_configs():
    """d=4096; k in {32,64,128}; N in {4096,16384,65536,131072}; Zipf(1.1) ids."""
    out = []
    i = 0
    for k in (32, 64, 128):
        for N in (4096, 16384, 65536, 131072):
            out.append(CodecConfig(f"sweep_k{k}_n{N}", B=1, S=N, d=4096, k=k, V=131072,
                                   dtype="bf16", seed=1005 + i, structured=False,
                                   ids_dist="zipf", zipf_s=1.1))
            i += 1
    return out


def paper_configs():
    """The paper's own stage-boundary shapes (section 5.2 model card and the
    1B ablation card of section 6): Pluralis-8B d=5120 at rank ~51 (100x),
    S=4096; the 1B model d=2048 at rank 40, S=2048; vocabulary 128,256; a
    microbatch of b coalesced sequences, b in {1, 2, 3}."""
    out = []
    for b in (1, 2, 3):
        out.append(CodecConfig(f"paper8b_b{b}", B=b, S=4096, d=5120, k=51, V=128256,
                               dtype="bf16", seed=1020 + b, structured=False))
    for b in (1, 2, 3):
        out.append(CodecConfig(f"paper1b_b{b}", B=b, S=2048, d=2048, k=40, V=128256,
                               dtype="bf16", seed=1024 + b, structured=False))
    return out


# Output projections of one body stage (4 layers) at the paper's shapes:
# W_o [d, d] and W_down [d, ffn] with ffn = d * 8/3 * 1.3 rounded up to a
# multiple of 1024 (18,432 at d=5120, 7,168 at d=2048).
WEIGHTS_PAPER8B = WeightsConfig("weights_paper8b", d=5120, k=51, layers=4,
                                shapes=((5120, 5120), (5120, 18432)), dtype="bf16", seed=1030)
WEIGHTS_PAPER1B = WeightsConfig("weights_paper1b", d=2048, k=40, layers=4,
                                shapes=((2048, 2048), (2048, 7168)), dtype="bf16", seed=1031)

CONFIGS = {c.name: c for c in [TINY, MID, STAGE8B] + sweep_configs() + paper_configs()}


@dataclasses.dataclass(frozen=True)
class SpartaConfig:
    """One sparse-averaging round over a block of float32 master weights."""
    name: str
    n: int                 # parameters of the block
    R: int                 # replicas contributing to the round
    seed: int
    segments: int = 20     # p = 1 / segments of the block per round
    std: float = 0.02      # weight scale
    drift: float = 1e-3    # spread between replicas, and local progress per round

    @property
    def m(self) -> int:
        return self.n // self.segments


# The paper's per-block estimate (section 4.2): p = 5% of a block is about 16M
# parameters, 0.5 Gbit per round against 10 Gbit for the whole block, so a
# block holds about 320M float32 parameters; four senders as in the averaging
# round pictured in section 3.3.1.
SPARTA_BLOCK8B = SpartaConfig("sparta_block8b", n=320_000_000, R=4, seed=1040)
SPARTA_TINY = SpartaConfig("sparta_tiny", n=100_003, R=3, seed=1041)


def sparta_replicas_host(n: int, R: int, seed: int, std: float = 0.02,
                         drift: float = 1e-3) -> np.ndarray:
    """[R, n] float32 replicas: a shared N(0, std^2) vector plus per-replica
    N(0, drift^2) divergence."""
    base = std * rng(seed, "theta").standard_normal(n)
    spread = drift * rng(seed, "drift").standard_normal((R, n))
    return (base[None, :] + spread).astype(np.float32)


def sparta_progress_host(n: int, seed: int, drift: float = 1e-3) -> np.ndarray:
    """[n] float32 local progress a replica makes while a round is in flight."""
    return (drift * rng(seed, "progress").standard_normal(n)).astype(np.float32)


def sparta_positions_host(n: int, m: int, seed: int, order: str = "sorted") -> np.ndarray:
    """m distinct int64 positions in [0, n): a shared random index set, sorted
    or in random order."""
    pos = rng(seed, "P").choice(n, size=m, replace=False).astype(np.int64)
    return np.sort(pos) if order == "sorted" else pos


def sparta_replica_device(n: int, seed: int, device, std: float = 0.02):
    """[n] float32 weights of one replica drawn on the device."""
    import torch
    return std * torch.randn(n, generator=_gen(device, seed, "theta"), device=device)


def sparta_chunks_device(snap, R: int, seed: int, drift: float = 1e-3):
    """R senders' chunks around a snapshot: chunk 0 is the snapshot itself,
    the others add N(0, drift^2) divergence (device draws)."""
    import torch
    g = _gen(snap.device, seed, "drift")
    out = [snap.clone()]
    for _ in range(R - 1):
        out.append(snap + drift * torch.randn(snap.shape, generator=g, device=snap.device))
    return out


def sparta_positions_device(n: int, m: int, seed: int, device):
    """m distinct sorted int64 positions in [0, n) drawn on the device."""
    import torch
    perm = torch.randperm(n, generator=_gen(device, seed, "P"), device=device)
    return torch.sort(perm[:m]).values.contiguous()


def with_tokens(cfg: CodecConfig, N: int, seed: Optional[int] = None) -> CodecConfig:
    """The same workload with a different token count (B=1, S=N)."""
    return dataclasses.replace(cfg, B=1, S=N, seed=cfg.seed if seed is None else seed)


def codec_inputs_host(cfg: CodecConfig, basis: str = "gaussian") -> Dict[str, np.ndarray]:
    """Host draws for a codec workload.

    Returns stored arrays U, E (dtype cfg.dtype), ids (int32), G (stored) and,
    for unstructured workloads, X (stored).  For structured workloads it returns
    the float64 draws Z0 (N x k) and eta (N x d); the caller composes
    X = E[ids] + Z0 U^T + eta with the codec oracle and rounds it once.
    U_f64 is the basis before rounding to the storage dtype.
    """
    if basis == "gaussian":
        u64 = gaussian_orthonormal_basis(cfg.d, cfg.k, cfg.seed)
    elif basis == "hadamard":
        u64 = hadamard_basis(cfg.d, cfg.k, cfg.seed)
    elif basis == "selection":
        u64 = selection_basis(cfg.d, cfg.k, cfg.seed)
    else:
        raise ValueError(basis)
    out = {
        "U_f64": u64,
        "U": store(u64, cfg.dtype),
        "E": store(cfg.emb_std * rng(cfg.seed, "E").standard_normal((cfg.V, cfg.d), dtype=np.float32),
                   cfg.dtype),
        "ids": token_ids(cfg.N, cfg.V, cfg.seed, cfg.ids_dist, cfg.zipf_s),
        "G": store(rng(cfg.seed, "G").standard_normal((cfg.N, cfg.d), dtype=np.float32), cfg.dtype),
    }
    if cfg.structured:
        out["Z0"] = rng(cfg.seed, "Z0").standard_normal((cfg.N, cfg.k))
        out["eta"] = cfg.noise_std * rng(cfg.seed, "noise").standard_normal((cfg.N, cfg.d))
    else:
        out["X"] = store(rng(cfg.seed, "X").standard_normal((cfg.N, cfg.d), dtype=np.float32),
                         cfg.dtype)
    return out


def coords_host(N: int, k: int, seed: int) -> np.ndarray:
    """float32 N(0,1) coordinates Z [N, k] (inputs of decompress / expansion)."""
    return rng(seed, "Z0").standard_normal((N, k), dtype=np.float32)


def weights_host(d: int, n: int, seed: int, dtype: str = "bf16", std: float = 0.02) -> np.ndarray:
    return store(std * rng(seed, "W").standard_normal((d, n), dtype=np.float32), dtype)


# --------------------------------------------------------------------------
# Device backend (torch).  Same distributions, drawn by torch's generator on
# the GPU.  Imported lazily so the host backend needs no torch.
# --------------------------------------------------------------------------
def _torch_dtype(dtype: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def _gen(device, seed: int, stream: str):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1009 + STREAM[stream])
    return g


def codec_inputs_device(cfg: CodecConfig, device, need=("U", "E", "ids", "X", "G")):
    """Device draws for an unstructured codec workload (X, G ~ N(0,1))."""
    import torch
    tdt = _torch_dtype(cfg.dtype)
    out = {}
    if "U" in need:
        u = store(gaussian_orthonormal_basis(cfg.d, cfg.k, cfg.seed), cfg.dtype)
        out["U"] = _host_to_device(u, cfg.dtype, device)
    if "E" in need:
        e = torch.empty((cfg.V, cfg.d), dtype=tdt, device=device)
        g = _gen(device, cfg.seed, "E")
        rows = max(1, (1 << 27) // cfg.d)      # draw in slabs to bound the fp32 temporary
        for r0 in range(0, cfg.V, rows):
            r1 = min(cfg.V, r0 + rows)
            e[r0:r1] = (cfg.emb_std * torch.randn((r1 - r0, cfg.d), generator=g, device=device)).to(tdt)
        out["E"] = e
    if "ids" in need:
        g = _gen(device, cfg.seed, "ids")
        if cfg.ids_dist == "uniform":
            out["ids"] = torch.randint(0, cfg.V, (cfg.N,), generator=g, device=device, dtype=torch.int32)
        else:
            cdf = torch.from_numpy(zipf_cdf(cfg.V, cfg.zipf_s)).to(device)
            u = torch.rand((cfg.N,), generator=g, device=device, dtype=torch.float64)
            rank = torch.clamp(torch.searchsorted(cdf, u, right=True), max=cfg.V - 1)
            perm = torch.randperm(cfg.V, generator=_gen(device, cfg.seed, "perm"), device=device)
            out["ids"] = perm[rank].to(torch.int32)
    for key in ("X", "G"):
        if key in need:
            g = _gen(device, cfg.seed, key)
            out[key] = torch.randn((cfg.N, cfg.d), generator=g, device=device).to(tdt)
    return out


def coords_device(N: int, k: int, seed: int, device):
    """float32 N(0,1) coordinates Z [N, k] drawn on the device."""
    import torch
    return torch.randn((N, k), generator=_gen(device, seed, "Z0"), device=device)


def weights_device(d: int, n: int, seed: int, device, dtype: str = "bf16", std: float = 0.02):
    import torch
    g = _gen(device, seed, "W")
    return (std * torch.randn((d, n), generator=g, device=device)).to(_torch_dtype(dtype))


def _host_to_device(a: np.ndarray, dtype: str, device):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def to_device(a: np.ndarray, dtype: str, device):
    """Stored host array (uint16 bf16 bits / float32 / int32) -> torch tensor on device."""
    import torch
    if a.dtype == np.int32:
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)
    return _host_to_device(a, dtype, device)


def to_host(t) -> np.ndarray:
    """torch tensor -> stored host array (bf16 as uint16 bits, others as is)."""
    import torch
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
