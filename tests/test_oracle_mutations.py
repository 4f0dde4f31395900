"""Plants plausible mistakes in a copy of the oracle's source (on the CPU, in a
temporary directory) and checks that the pins catch every one of them: a pin
set that a dropped term, a swapped operand or an off-by-one slips through
would not be pinning anything."""
import ctypes as C
import os
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
from oracle import build as obuild
from synth import meshes
import torch_ref
from cases import local_case

SRC = os.path.join(os.path.dirname(obuild.LIB), "mgn_oracle.cpp")

MUTATIONS = {
    "edge_residual_dropped": ("e_next[ed * l + i] = Q.r(e[ed * l + i] + msg[ed * l + i]);",
                              "e_next[ed * l + i] = Q.r(msg[ed * l + i]);"),
    "sender_receiver_swapped": ("x[l + i] = v[s * l + i];\n      x[2 * l + i] = v[r * l + i];",
                                "x[l + i] = v[r * l + i];\n      x[2 * l + i] = v[s * l + i];"),
    "unbiased_variance": ("  var /= n;", "  var /= (n - 1);"),
    "node_residual_dropped": ("v_next[r * l + i] = v[r * l + i] + y[i];", "v_next[r * l + i] = y[i];"),
    "weight_transposed": ("const double* w = Q.W + L.w + (int64_t)o * L.in;\n      for (int i = 0; i < L.in; ++i) s += w[i] * t.a[j][i];",
                          "for (int i = 0; i < L.in; ++i) s += Q.W[L.w + (int64_t)i * L.out + (o % L.in)] * t.a[j][i];"),
    "halo_block_off_by_one": ("halo[((int64_t)k * n_halo + h) * l + i]",
                              "halo[((int64_t)(k + 1 < K ? k + 1 : k) * n_halo + h) * l + i]"),
    "dagg_dropped": ("dm[i] = de[ed * l + i] + dagg[r * l + i];", "dm[i] = de[ed * l + i];"),
    "ln_backward_mean_term_dropped": ("dz[o] = t.rstd * (dxh[o] - mean_d - t.xhat[o] * mean_dx);",
                                      "dz[o] = t.rstd * (dxh[o] - t.xhat[o] * mean_dx);"),
    "relu_mask_on_output": ("dz[i] = t.z[j - 1][i] > 0 ? da[i] : 0.0;", "dz[i] = da[i];"),
    "edge_feature_sign": ("d[a] = (coords[3 * (int64_t)send[e] + a] - coords[3 * (int64_t)recv[e] + a]) / h;",
                          "d[a] = (coords[3 * (int64_t)recv[e] + a] - coords[3 * (int64_t)send[e] + a]) / h;"),
    "halo_grad_dropped": ("for (int i = 0; i < l; ++i) dh[i] += dxs[ed * l + i];", "(void)dh;"),
    "halo_ordered_after_owned_wrongly": ("if (is_halo[g]) g2l[g] = next++;", "if (is_halo[g]) g2l[g] = next++ ^ 1;"),
    "edge_gradient_not_rounded_in_bf16": ("de_next[ed * l + i] = Q.r(de[ed * l + i] + dx[i]);",
                                          "de_next[ed * l + i] = de[ed * l + i] + dx[i];"),
}


def _compile(tmp, name, src):
    path = os.path.join(tmp, f"{name}.cpp")
    with open(path, "w") as f:
        f.write(src)
    lib = os.path.join(tmp, f"lib{name}.so")
    subprocess.run(["g++", "-O1", "-std=c++17", "-fopenmp", "-fPIC", "-shared", "-I", os.path.dirname(SRC),
                    path, "-o", lib], check=True)
    return lib


def _pins_pass():
    """A compact run of the oracle pins; False as soon as one fails."""
    try:
        c = local_case(meshes.sector(3, 8, 4, 4, seed=2), 1, 8, 2, 3, seed=3)
        g = c["g"]
        r = oracle.step(c["cfg"], g, c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
        out, dp, dh = torch_ref.run(8, 2, 3, c["shapes"], g, c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
        if not (np.allclose(r["out"], out, atol=1e-10) and np.allclose(r["d_params"], dp, atol=1e-9)
                and np.allclose(r["d_halo"], dh, atol=1e-9)):
            return False
        # the mixed-precision mode against torch's bfloat16 rounding at the same points
        cb = oracle.ModelCfg(8, 2, 3, bf16=True)
        rb = oracle.step(cb, g, c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
        out, dp, dh = torch_ref.run(8, 2, 3, c["shapes"], g, c["params"], c["nf"], c["ef"], c["halo"], c["d_out"],
                                    bf16=True)
        if not (np.allclose(rb["out"], out, atol=1e-10) and np.allclose(rb["d_params"], dp, atol=1e-9)
                and np.allclose(rb["d_halo"], dh, atol=1e-9)):
            return False
        m = meshes.sector(4, 12, 5, 4, seed=1)
        if not np.allclose(oracle.edge_features(m.coords, m.send, m.recv, m.h),
                           (lambda d: np.concatenate([d, np.linalg.norm(d, axis=1, keepdims=True)], 1))(
                               (m.coords[m.send] - m.coords[m.recv]) / m.h)):
            return False
        from cases import brute_graph
        part = oracle.partition(m.key, 4)
        gb = oracle.graph_build(m.send, m.recv, part, m.n_nodes, 1)
        bb = brute_graph(m.send, m.recv, part, m.n_nodes, 1)
        return all(np.array_equal(np.asarray(gb[k]), np.asarray(bb[k])) for k in bb)
    except (ValueError, IndexError):
        return False


def test_every_planted_mistake_is_caught():
    src = open(SRC).read()
    caught, missed = [], []
    saved = oracle._lib
    with tempfile.TemporaryDirectory() as tmp:
        try:
            for name, (a, b) in MUTATIONS.items():
                assert src.count(a) == 1, f"mutation anchor for {name} not unique in the oracle source"
                oracle._lib = None
                lib = C.CDLL(_compile(tmp, name, src.replace(a, b)))
                lib.orc_param_count.restype = C.c_int64
                oracle._lib = lib
                (missed if _pins_pass() else caught).append(name)
            oracle._lib = None
            lib = C.CDLL(_compile(tmp, "unmutated", src))
            lib.orc_param_count.restype = C.c_int64
            oracle._lib = lib
            assert _pins_pass(), "the unmutated oracle must pass"
        finally:
            oracle._lib = saved
    assert not missed, f"pins missed planted mistakes: {missed}"
