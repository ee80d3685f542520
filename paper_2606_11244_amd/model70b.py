"""The 70B-shaped model's linear layers resident on the GPU: 80 layers x 7
modules of group-128 int4 weights with device-random codes, scales and zero
points (about 36 GB), and the EC (rank 64, sigmoid-linear gate, fp16) on the
seeded quarter of the (layer, module) pairs. Timing-only weights: the
benchmark's whole-model pass and the sampled full-model parity test build it
here the same way."""
from __future__ import annotations

RANK, GROUP = 64, 128


def build(device="cuda", seed=0, layers=None, weight_bits=4):
    """Returns (modules, selection): modules[l][j] = (name, K, N, qweight
    int32 [N][K/8] (3-bit codes: [N][3K/32]), scales fp16 bits as int16
    [N][K/128], zeros uint8 [N][K/128], ec) with ec = (A [64][K], B [N][64],
    w_g [K]) fp16 on the selected pairs, else None; selection is the bool
    [80][7] EC choice."""
    import torch

    from paper_2606_11244_amd import synth as S
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    sel = S.ec_selection_70b(seed=seed)
    n_layers = sel.shape[0] if layers is None else layers
    out = []
    for l in range(n_layers):
        mods = []
        for j, m in enumerate(S.MODULES):
            K, N = S.LLAMA_70B[m]
            q = torch.randint(-2**31, 2**31 - 1, (N, K // 8 if weight_bits == 4 else K // 32 * 3),
                              dtype=torch.int32, device=device, generator=g)
            sc = (torch.rand((N, K // GROUP), device=device, generator=g) * 1e-3 + 1e-4).half()
            zr = torch.randint(0, 1 << weight_bits, (N, K // GROUP), dtype=torch.uint8,
                               device=device, generator=g)
            ec = None
            if sel[l, j]:
                ec = ((torch.randn((RANK, K), device=device, generator=g) * 0.01).half(),
                      (torch.randn((N, RANK), device=device, generator=g) * 0.01).half(),
                      (torch.randn((K,), device=device, generator=g) * 0.05).half())
            mods.append((m, K, N, q, sc.view(torch.int16), zr, ec))
        out.append(mods)
    return out, sel
