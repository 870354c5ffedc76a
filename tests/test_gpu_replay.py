"""GPU parity of the open-loop replay (ssmq_replay) against the oracle's replay
(Appendix B "Open-loop replay"), through the C ABI: codes, scales and final
reference states bit for bit, and the per-block error sums equal, since both
sides form and add the same double terms in the same order."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def ssmq():
    import paper_2609_39185_amd as m
    m.library()
    return m


def _traces(n, T, seed):
    """Decays spanning short and long memories (a in [0.5, 1], some exactly 1 and
    0), writes of mixed magnitude (some tiny, some zero), and an h0 with zeros,
    tiny values and a wide range of magnitudes."""
    rng = np.random.default_rng(seed)
    tau = np.exp(rng.uniform(0.0, np.log(3000.0), n))
    a = np.exp(-rng.uniform(0.5, 1.5, (T, n)) / tau).astype(np.float32)
    a[:, ::97] = 1.0
    a[T // 2, ::53] = 0.0
    w = (rng.standard_normal((T, n)) * np.exp(rng.uniform(-12, 0, n))).astype(np.float32)
    w[:, ::61] = 0.0
    w[:, 5::89] *= np.float32(1e-30)
    h0 = (rng.standard_normal(n) * np.exp(rng.uniform(-8, 4, n))).astype(np.float32)
    h0[::71] = 0.0
    h0[3::83] = np.float32(-1e-39)
    return h0, a, w


def _run(ssmq, fmt, rule, h0, a, w, group, block_steps, **q):
    n, T = h0.size, a.shape[0]
    nb = (T + block_steps - 1) // block_steps
    per = oracle.entries_per_code_word(fmt)
    dt = {"fp16": torch.int16, "bf16": torch.int16, "e4m3": torch.uint8, "fp32": torch.int32,
          "int8": torch.uint8, "int4": torch.uint8}[fmt]
    err = torch.full((nb, n), -1.0, dtype=torch.float64, device=DEV)
    ref = torch.full((nb, n), -1.0, dtype=torch.float64, device=DEV)
    codes = torch.zeros(n // per, dtype=dt, device=DEV)
    scale = torch.zeros(max(n // group, 1), device=DEV) if group else None
    hf = torch.zeros(n, device=DEV)
    ssmq.replay(torch.from_numpy(h0).to(DEV), torch.from_numpy(a).to(DEV),
                torch.from_numpy(w).to(DEV), err, rule=rule, fmt=fmt, ref=ref, codes=codes,
                scale=scale, h_final=hf, block_steps=block_steps, scale_group=group, **q)
    torch.cuda.synchronize()
    got = {"err": err.cpu().numpy(), "ref": ref.cpu().numpy(),
           "codes": codes.cpu().numpy().view(oracle.CODE_DTYPE[fmt]),
           "scale": None if scale is None else scale.cpu().numpy(), "h_final": hf.cpu().numpy()}
    want = oracle.replay(fmt, rule, h0, a, w, group=group, block_steps=block_steps,
                         **{("block" if k == "dither_block" else k): v for k, v in q.items()})
    return got, want


def _same(got, want, what):
    for k in ("codes", "h_final", "err", "ref"):
        assert np.array_equal(got[k], want[k], equal_nan=True), (what, k)
    if want["scale"] is not None:
        assert np.array_equal(got["scale"], want["scale"]), (what, "scale")


FORMATS = [("fp16", 0), ("bf16", 0), ("e4m3", 16), ("int8", 16), ("int4", 16), ("fp32", 0)]


@pytest.mark.parametrize("fmt,group", FORMATS)
@pytest.mark.parametrize("rule", ["rtn", "sr", "weyl", "philox"])
def test_replay_matches_oracle(ssmq, fmt, group, rule):
    # 197 groups of 16: three full workgroups of 256 threads and a ragged fourth
    n, T = 16 * 197, 37
    h0, a, w = _traces(n, T, seed=10 * [f for f, _ in FORMATS].index(fmt)
                       + ["rtn", "sr", "weyl", "philox"].index(rule))
    say(f"case replay {fmt} {rule}: n {n}, T {T}, blocks of 8 steps")
    got, want = _run(ssmq, fmt, rule, h0, a, w, group, 8, dither_block=16, seed=3, layer=7,
                     step=500, entry_base=4096)
    _same(got, want, (fmt, rule))


@pytest.mark.parametrize("fmt,group", [("int8", 128), ("e4m3", 256), ("int4", 4), ("bf16", 0)])
def test_replay_groups_and_blocks(ssmq, fmt, group):
    """Groups that span 32 and 64 lanes or one lane, the hybrids' dither block of 128."""
    n, T = 256 * 41, 20
    h0, a, w = _traces(n, T, seed=5)
    say(f"case replay {fmt} group {group}: n {n}, T {T}")
    got, want = _run(ssmq, fmt, "weyl", h0, a, w, group, 6, dither_block=128, seed=0, layer=1,
                     step=2 ** 32 - 3)   # the step counter wraps mid-replay
    _same(got, want, (fmt, group))


def test_replay_without_steps_and_optional_outputs(ssmq):
    n = 1024
    h0, a, w = _traces(n, 1, seed=8)
    got, want = _run(ssmq, "int8", "sr", h0, a[:0], w[:0], 16, 4)   # T = 0: Q_0 alone
    assert got["err"].size == 0
    _same(got, want, "T = 0")
    # only err requested
    err = torch.zeros((1, n), dtype=torch.float64, device=DEV)
    ssmq.replay(torch.from_numpy(h0).to(DEV), torch.from_numpy(a).to(DEV),
                torch.from_numpy(w).to(DEV), err, rule="sr", fmt="int8", scale_group=16)
    torch.cuda.synchronize()
    want = oracle.replay("int8", "sr", h0, a, w, group=16)
    assert np.array_equal(err.cpu().numpy(), want["err"])


def test_replay_full_layer_sampled(ssmq):
    """A Mamba-1 layer of the long-horizon shape (batch 16 x d_inner 5120 x N 16 =
    1,310,720 entries), 64 steps, INT8 blocks of 16 under Weyl: sampled ranges of
    entries replayed by the oracle with their global entry_base."""
    n, T = 16 * 5120 * 16, 64
    h0, a, w = _traces(n, T, seed=12)
    say(f"case replay full layer: n {n}, T {T}")
    err = torch.zeros((T // 16, n), dtype=torch.float64, device=DEV)
    codes = torch.zeros(n, dtype=torch.uint8, device=DEV)
    scale = torch.zeros(n // 16, device=DEV)
    ssmq.replay(torch.from_numpy(h0).to(DEV), torch.from_numpy(a).to(DEV),
                torch.from_numpy(w).to(DEV), err, rule="weyl", fmt="int8", codes=codes,
                scale=scale, block_steps=16, scale_group=16, layer=9, step=77)
    torch.cuda.synchronize()
    err, codes, scale = err.cpu().numpy(), codes.cpu().numpy(), scale.cpu().numpy()
    for lo in (0, 655360, n - 4096):
        sl = slice(lo, lo + 4096)
        want = oracle.replay("int8", "weyl", h0[sl], a[:, sl], w[:, sl], group=16, block_steps=16,
                             layer=9, step=77, entry_base=lo)
        assert np.array_equal(err[:, sl], want["err"])
        assert np.array_equal(codes[sl], want["codes"])
        assert np.array_equal(scale[lo // 16:(lo + 4096) // 16], want["scale"])
