"""GPU: lc_score_layers_static, the score for callers that cannot allocate,
against lc_score_layers on the same weights and shadow (bit for bit) and the
oracle's Eq. 1 (within 1e-5), on calls in a row through the one fixed device
array: the full Llama-3-8B-shaped weights and shadow (16 GB each, scored in
three batches of whole layers), then the smaller reduced 8B layout, then the
fp32 toy decoder."""
import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import inputs as I
from paper_2609_27193_amd import layercheck as LC
from tests.conftest import gpu_available
from tests.gpu_harness import REL, log, rel_ok

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    LC.load_library()


class WS:
    """Weights and shadow of a spec's layout, flat on the device; the shadow
    equals the weights (as lc_init_layout leaves it) until ``perturb``."""

    def __init__(self, spec, seed):
        import torch
        self.spec = spec
        self.N = spec.n_layers
        dt = torch.bfloat16 if spec.weight_dtype == "bf16" else torch.float32
        self.dtype = LC.LC_DT_BF16 if spec.weight_dtype == "bf16" else LC.LC_DT_F32
        self.sizes = [[t.numel for t in l.tensors] for l in spec.layers]
        total = sum(sum(s) for s in self.sizes)
        self.W = torch.empty(total, dtype=dt, device="cuda")
        self.S = torch.empty(total, dtype=dt, device="cuda")
        self.gen = torch.Generator(device="cuda")
        self.gen.manual_seed(seed)
        self.segs, self.layer_slices, off = [], [], 0
        for l, layer in enumerate(self.sizes):
            a = off
            for n in layer:
                self.W[off:off + n] = torch.randn(n, generator=self.gen, device="cuda") * 0.02
                self.segs.append(LC.Segment(l, n, self.W[off:off + n].data_ptr(), self.S[off:off + n].data_ptr(),
                                            None, None, None))
                off += n
            self.layer_slices.append((a, off))
        self.S.copy_(self.W)

    def perturb(self):
        """Per-layer scaled change of the weights (update scales over two decades)."""
        import torch
        scales = torch.logspace(-2, 0, self.N, device="cpu").tolist()
        for l, (a, b) in enumerate(self.layer_slices):
            d = torch.randn(b - a, generator=self.gen, device="cuda") * (1e-3 * scales[l])
            self.W[a:b] = (self.W[a:b].float() + d).to(self.W.dtype)

    def host(self, l):
        a, b = self.layer_slices[l]
        to = I.to_numpy_weight
        return to(self.W[a:b].cpu()), to(self.S[a:b].cpu())


def run_case(spec, seed, oracle_layers):
    import torch
    ws = WS(spec, seed)
    stream = torch.cuda.current_stream().cuda_stream
    layout = LC.LayoutDesc(ws.segs, ws.N, ws.dtype, False, LC.LC_MODE_ACCUM, [float("inf")] * ws.N, 1 << 20,
                           stream=stream)
    ctx = LC.lc_init_layout(layout)  # S <- W
    try:
        ws.perturb()
        torch.cuda.synchronize()
        hosts = {l: ws.host(l) for l in oracle_layers}
        u_dev = torch.full((ws.N,), float("nan"), dtype=torch.float64, device="cuda")
        LC.lc_score_layers_static(ws.segs, ws.N, ws.dtype, 1e-8, u_dev.data_ptr(), stream)
        u_static = u_dev.cpu().numpy()
        s_before = ws.S.clone() if ws.S.numel() < (1 << 28) else None
        LC.lc_score_layers_static(ws.segs, ws.N, ws.dtype, 1e-8, u_dev.data_ptr(), stream)  # again: same bits
        assert np.array_equal(u_dev.cpu().numpy().view(np.uint64), u_static.view(np.uint64))
        if s_before is not None:
            assert torch.equal(ws.S.view(torch.uint8), s_before.view(torch.uint8))
        LC.lc_score_layers(ctx, 1)  # the context's score of the same W and S (ACCUM: then S <- W)
        u_ctx = LC.lc_read_state(ctx, ws.N)[0]
        assert np.array_equal(u_static.view(np.uint64), u_ctx.view(np.uint64)), (u_static, u_ctx)
        odt = O.DT_BF16 if ws.dtype == LC.LC_DT_BF16 else O.DT_F32
        for l in oracle_layers:
            w, s = hosts[l]
            uo = O.layer_update_score([w], [s], odt, 1e-8)[3]
            assert rel_ok([u_static[l]], [uo]) and u_static[l] > 0, (l, u_static[l], uo)
        log(f"  {spec.name}: {ws.N} layers, {ws.W.numel()} weights; u in [{u_static.min():.3e}, "
            f"{u_static.max():.3e}], bit-identical to lc_score_layers; oracle layers {list(oracle_layers)}")
    finally:
        LC.lc_destroy(ctx)
        del ws
        torch.cuda.empty_cache()


def test_static_score_matches_context_score_on_calls_in_a_row():
    from tests.test_parity_gpu import reduced_8b
    full = I.llama3_8b_spec()
    names = [l.name for l in full.layers]
    # 1.96 M score chunks: more than one batch of the 16 MiB array holds
    run_case(full, 11, [names.index("norm"), names.index("block_5")])
    small = reduced_8b()  # a smaller input: one batch, the array holding the previous call's tables
    run_case(small, 12, list(range(small.n_layers)))
    toy = I.toy_spec()  # fp32 weights
    run_case(toy, 13, list(range(toy.n_layers)))


def test_static_score_argument_errors():
    import torch
    from tests.test_parity_gpu import reduced_8b
    ws = WS(reduced_8b(), 14)
    u = torch.empty(ws.N, dtype=torch.float64, device="cuda")

    def expect(code, segs, n_layers, dtype=ws.dtype, u_ptr=None):
        with pytest.raises(LC.LCError) as e:
            LC.lc_score_layers_static(segs, n_layers, dtype, 1e-8, u.data_ptr() if u_ptr is None else u_ptr,
                                      torch.cuda.current_stream().cuda_stream)
        assert e.value.code == code, str(e.value)

    expect(LC.LC_ERR_INVALID_ARG, ws.segs, ws.N + 1)              # a layer with no segment
    expect(LC.LC_ERR_INVALID_ARG, ws.segs[::-1], ws.N)            # not grouped by ascending layer
    expect(LC.LC_ERR_INVALID_ARG, ws.segs, ws.N, dtype=7)         # unknown dtype
    host = np.zeros(ws.N)
    expect(LC.LC_ERR_INVALID_ARG, ws.segs, ws.N, u_ptr=host.ctypes.data)  # u_out in host memory
