"""The layer on a side stream and under HIP graph capture: the
allocation-free entry point (whose callers include code under capture) and
the workspace entry point, captured once and replayed several times, with
other eager calls of the library between the replays (they leave their own
data in the shared scratch and workspace) and a synchronisation before
each check.  Every replay must equal the eager result bit for bit: the
calls enqueue only kernels (counters are cleared by kernels, never by a
memset), allocate nothing and make no host synchronisation."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _layer(T, K, N, r, M, seed):
    from oracle.bf16 import bf16_round
    rng = np.random.default_rng(seed)
    counts = [T // M + (1 if m < T % M else 0) for m in range(M)]
    mod = synth.make_modality_layout(counts, "runs" if T >= 256 else "alternating", 0, seed)
    x = bf16_round(rng.standard_normal((T, K)).astype(np.float32) *
                   np.where(mod == 0, 1.0, 30.0).astype(np.float32)[:, None])
    return dict(x=x, modality=mod, inv_smooth=rng.uniform(0.05, 3.0, (M, K)).astype(np.float32),
                wq=rng.integers(-127, 128, (N, K)).astype(np.int8),
                w_scale=rng.uniform(1e-4, 1e-2, N).astype(np.float32),
                l_down=bf16_round((rng.standard_normal((M - 1, r, K)) / np.sqrt(K)).astype(np.float32)),
                r_up=bf16_round((rng.standard_normal((M - 1, N, r)) * 0.05).astype(np.float32)),
                n_mod=M, rank=r, act_dtype="bf16", lr_dtype="bf16", weight_bits=8)


_SHAPES = {
    "persistent_t4096_k3584_n2048": (4096, 3584, 2048, 64, 2),
    "split_k_t700_k1024_n528": (700, 1024, 528, 64, 3),
    "decode_t16_k4096_n512": (16, 4096, 512, 64, 2),
}


def _bits(y):
    return y.view(torch.int16).clone()


@pytest.mark.parametrize("name", list(_SHAPES))
def test_graph_replays_equal_eager(name):
    assert torch.cuda.is_available()
    from paper_2603_04800_amd import workload
    T, K, N, r, M = _SHAPES[name]
    x, mod, lin = workload.to_device(_layer(T, K, N, r, M, seed=41))
    # another layer whose eager calls run between the replays
    x2, mod2, lin2 = workload.to_device(_layer(300, 512, 256, 32, 3, seed=42))
    y2 = torch.empty((300, 256), dtype=torch.bfloat16, device=x.device)
    print(f"[graph] {name}", flush=True)
    ref = _bits(lin(x, mod, out_dtype=torch.bfloat16))
    torch.cuda.synchronize()

    ws = lin.workspace(T, x.device)
    y_na = torch.empty((T, N), dtype=torch.bfloat16, device=x.device)
    y_ws = torch.empty((T, N), dtype=torch.bfloat16, device=x.device)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):           # warm-up and a side-stream check
        lin.noalloc(x, mod, y_na)
        lin(x, mod, out=y_ws, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert torch.equal(_bits(y_na), ref) and torch.equal(_bits(y_ws), ref), "side stream"

    g_na, g_ws = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_na):
        lin.noalloc(x, mod, y_na)
    with torch.cuda.graph(g_ws):
        lin(x, mod, out=y_ws, workspace=ws)
    torch.cuda.synchronize()
    for rep in range(3):
        y_na.fill_(float("nan"))
        y_ws.fill_(float("nan"))
        lin2.noalloc(x2, mod2, y2)          # eager work on the shared scratch
        lin2(x2, mod2, out=y2, workspace=ws if ws.numel() >= _need(lin2) else None)
        torch.cuda.synchronize()
        g_na.replay()
        torch.cuda.synchronize()
        assert torch.equal(_bits(y_na), ref), f"{name}: noalloc replay {rep}"
        g_ws.replay()
        torch.cuda.synchronize()
        assert torch.equal(_bits(y_ws), ref), f"{name}: workspace replay {rep}"


def _need(lin):
    from paper_2603_04800_amd import ops
    return ops.workspace_bytes(300, lin.c_in, lin.c_out, lin.rank, lin.n_mod)


def test_concurrent_streams_with_separate_workspaces():
    """Two layers (tiled and split-K shapes) on two streams at the default
    priority, each with its own workspace, enqueued interleaved so that their
    kernels can overlap: the workspace entry point keeps no state outside its
    workspace, so each result equals its sequential one bit for bit."""
    assert torch.cuda.is_available()
    from paper_2603_04800_amd import ops, workload
    layers = [workload.to_device(_layer(*_SHAPES[n], seed=50 + i))
              for i, n in enumerate(("persistent_t4096_k3584_n2048", "split_k_t700_k1024_n528"))]
    refs = [_bits(lin(x, mod, out_dtype=torch.bfloat16)) for x, mod, lin in layers]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs, wss = [], []
    for x, mod, lin in layers:
        outs.append(torch.empty((x.shape[0], lin.c_out), dtype=torch.bfloat16, device=x.device))
        need = ops.workspace_bytes(x.shape[0], lin.c_in, lin.c_out, lin.rank, lin.n_mod)
        wss.append(torch.empty(max(need, 256), dtype=torch.uint8, device=x.device))
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    for rep in range(4):
        for i, (x, mod, lin) in enumerate(layers):
            with torch.cuda.stream(streams[i]):
                lin(x, mod, out=outs[i], workspace=wss[i])
    torch.cuda.synchronize()
    for i in range(2):
        assert torch.equal(_bits(outs[i]), refs[i]), f"layer {i}"
