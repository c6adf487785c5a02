"""Full-size GPU checks at the workloads' real shapes.

Each workload runs the whole reconstruction: the source's full prefill of
every request, the pack of each suffix, the target's varlen prefix prefill,
the assembly of the suffix chunks and one batched decode step over the
assembled caches.

* Properties at full depth: for every layer the target's prefix K/V equal
  the source's unmigrated K/V bit for bit (causality), the assembled suffix
  equals the source's bit for bit, and the decode over the assembled caches
  gives the logits of the decode over the unmigrated ones, bit for bit.
* Oracle parity, layer-local.  The oracle cannot follow 36 or 64 layers at
  these sizes, and with depth the bf16 rounding decisions of a float32
  evaluation and a float64 one drift apart, so each sampled layer l is
  checked from the GPU's own input to it.  A model handle over the first
  l + 1 layers (the same weight tensors) prefills the same ids; its last
  layer runs only the K/V projection, so its workspace's residual section
  then holds the float32 residual the GPU feeds layer l (pallas.h).  The
  oracle runs layer l from that input: its K and V must match the GPU's
  layer-l K/V within 1e-2 max|ref| per tensor, and the residual update the
  layer adds (the next layer's input, from a model over l + 2 layers, minus
  this one's) within 1e-2 of the oracle's max.
* Decode, the same way over the assembled cache: the oracle's final norm
  and lm_head applied to the GPU decode's final residual give the logits
  within 1e-2 per row, and at sampled layers the oracle's decode layer,
  from the GPU decode's input to it and over the GPU's cache of that layer,
  gives the K/V the step writes and the residual update.

Large workload: 64 layers, hidden 5120, 64/8 heads, ffn 25600; one request
of 4000 tokens split at 3000 (one suffix chunk); layers 0, 1, 31, 62, 63 over
all 3000 positions; decode at position 4000.
Mid workload: 36 layers, hidden 4096, 32/8 heads, ffn 12288; one request of
2048 split at 1536; layers 0, 8, 17, 26, 35 over all 1536 positions.
Concurrent workload: the mid model, 8 requests of 1000-8000 tokens in
32-token suffix chunks; K/V of layers 0, 17, 35 over every prefix position,
the residual update on the last 64 rows of each request; the 8-row decode
batch."""
import numpy as np
import pytest
import torch

from helpers import TOL, ensure_lib, rel_err, to_np64
from oracle import model as om
from oracle import numerics as on
from recon import Recon
from workloads import configs

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
DEV = "cuda"


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


@pytest.fixture(scope="module")
def large(P):
    return Recon(P, configs.workload("large"))


@pytest.fixture(scope="module")
def mid(P):
    return Recon(P, configs.workload("mid"))


@pytest.fixture(scope="module")
def concurrent(P):
    return Recon(P, configs.workload("concurrent"))


def test_large_properties(large):
    large.check_properties()


@pytest.mark.parametrize("layer", [0, 1, 31, 62, 63])
def test_large_prefill_layer_local(large, layer):
    large.check_prefill_layer(layer)


def test_large_decode_layer_local(large):
    large.check_decode([0, 31, 63])


def test_mid_properties(mid):
    mid.check_properties()


@pytest.mark.parametrize("layer", [0, 8, 17, 26, 35])
def test_mid_prefill_layer_local(mid, layer):
    mid.check_prefill_layer(layer)


def test_mid_decode_layer_local(mid):
    mid.check_decode([0, 17, 35])


def test_mid_full_depth_report(mid):
    """Full-depth oracle on positions [0, 48), as a report of how the error
    against a float64 evaluation of the whole depth grows: the first four
    layers must meet 1e-2 max|ref|; deeper layers are printed next to the
    drift of the oracle's own float32 evaluation (bf16 at the same points)
    from its float64 one, which grows the same way.  Parity of every layer
    at 1e-2 is what the layer-local tests check."""
    r, t = mid, 48
    ids = torch.as_tensor(r.ids[0][:t], dtype=torch.long, device=DEV)
    emb = to_np64(r.glob["embed"][ids])
    r64, r32 = emb, emb.astype(np.float32)
    pos = np.arange(t)
    errs, drift, worst = [], [], 0.0
    for l in range(r.cfg.n_layers):
        w = r.lazy[l]
        last = l == r.cfg.n_layers - 1
        r64, k64, v64 = om.layer(r64, pos, None, None, w, r.shp, om.bf16_round, kv_only=last)
        with om.precision(np.float32):
            w32 = {k: v.astype(np.float32) for k, v in w.items()}
            r32, k32, v32 = om.layer(r32, pos, None, None, w32, r.shp, on.bf16_round_as, kv_only=last)
        worst = max(worst, rel_err(k32, k64), rel_err(v32, v64))
        drift.append(worst)
        got = r.kv(r.dst, r.dst_tab, 0, t, l)
        errs.append(max(rel_err(got[0], k64), rel_err(got[1], v64)))
    print("layer: gpu rel err against the full-depth oracle / oracle float32 drift:",
          " ".join(f"{l}:{e:.4f}/{d:.4f}" for l, (e, d) in enumerate(zip(errs, drift))))
    for l in range(4):
        assert errs[l] <= TOL, f"layer {l}: {errs[l]:.3g}"


def test_concurrent_properties(concurrent):
    concurrent.check_properties()


@pytest.mark.parametrize("layer", [0, 17, 35])
def test_concurrent_prefill_layer_local(concurrent, layer):
    concurrent.check_prefill_layer(layer, tail=64)


def test_concurrent_decode_layer_local(concurrent):
    concurrent.check_decode([0, 35])
