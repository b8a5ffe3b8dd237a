"""GPU parity of the decode-time exit decision (ee_exit_decide) against the
fp64 oracle (oracle/decode.py).

The device rounds what the output matrix sees (Z) to the exit's dtype, as in
training, so each logit may differ from the oracle's by at most
    E_v = c * sum_k |W_out[v, k]| |z_k|,
with c = 2^-8 for a bf16 Norm exit (one bf16 rounding of z, 2x margin),
2^-6 for a bf16 MLP exit (roundings of U, H_g, A and z, 2x margin), 2^-20
for fp32 and for the Embedding exit (fp32 accumulation only).  With
E = max_v E_v per row:
  * token: equal to the oracle's when the oracle's top-2 gap exceeds 2E;
    otherwise its oracle logit must be within 2E of the maximum;
  * confidence: |log c_gpu - log c_oracle| <= 2E + 1e-5;
  * exit flag: equal wherever |log c_oracle - log threshold| exceeds that bound.
"""

import numpy as np
import pytest
import torch

import oracle as O
from oracle import decode as D
import workloads as W
from paper_2402_00518_amd import binding as B
from paper_2402_00518_amd.session import to_device

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)


def make_case(kind, n, h, V, I, dtype, seed, norm="rms", bias=False):
    w = W.custom(kind, n, h, V, I, dtype, (1.0,), row_scale=True, zipf=True, name="decode",
                 norm=norm, bias=bias)
    b = W.make_batch(w, seed, random_gamma=True)
    return w, b


def run_decide(b, threshold, dev_params=None):
    w = b.workload
    p = b.exits[0]
    d = {"w_out": p.w_out, "gamma": p.gamma, "gamma_mlp": p.gamma_mlp, "w_gate": p.w_gate,
         "w_up": p.w_up, "w_down": p.w_down, "beta": p.beta}
    t = dev_params or {k: to_device(a, "cuda") for k, a in d.items() if a is not None}
    dtype = B.EE_F32 if w.dtype == "f32" else B.EE_BF16
    inter = w.intermediate if w.kind == B.EE_EXIT_MLP else 0
    norm = B.EE_NORM_LAYER if w.norm == "layer" else B.EE_NORM_RMS
    e = B.make_exit(w.kind, dtype, w.hidden, w.vocab, inter, w.eps, norm=norm, **t)
    n = w.n_tokens
    x = to_device(b.hidden[0], "cuda")
    ws_bytes = B.ee_decode_workspace_bytes(e, n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    token = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    conf = torch.full((n,), -1.0, dtype=torch.float32, device="cuda")
    flag = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    B.ee_exit_decide(e, x, n, threshold, token, conf, flag, ws, ws_bytes, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return token.cpu().numpy(), conf.cpu().numpy().astype(np.float64), flag.cpu().numpy()


def check(b, threshold, got):
    w = b.workload
    ex = O.exits_from_batch(b)[0]
    x = W.decode(b.hidden[0])
    ref = D.exit_decide(ex, x, threshold)
    z = O.exit_forward(ex, x)["z"]
    if w.dtype == "f32" or w.kind == W.EXIT_EMBEDDING:
        c = 2.0 ** -20
    elif w.kind == W.EXIT_MLP:
        c = 2.0 ** -6
    else:
        c = 2.0 ** -8
    E = c * (np.abs(z) @ np.abs(ex.w_out).T).max(axis=1)      # per row
    token, conf, flag = got
    s = ref["logits"]
    n = s.shape[0]
    assert ((flag == 0) | (flag == 1)).all()
    assert ((token >= 0) & (token < w.vocab)).all()
    if w.vocab > 1:
        top2 = np.sort(s, axis=1)[:, -2:]
        gap = top2[:, 1] - top2[:, 0]
    else:
        gap = np.full(n, np.inf)
    for r in range(n):
        if gap[r] > 2 * E[r]:
            assert token[r] == ref["token"][r], (r, token[r], ref["token"][r], gap[r], E[r])
        else:
            assert s[r, token[r]] >= s[r].max() - 2 * E[r], r
    bound = 2 * E + 1e-5
    err = np.abs(np.log(conf) - np.log(ref["confidence"]))
    assert (err <= bound).all(), (err.max(), bound[np.argmax(err - bound)])
    decided = np.abs(np.log(ref["confidence"]) - np.log(threshold)) > bound
    assert (flag[decided] == ref["exit"][decided].astype(np.int32)).all()
    return ref


CASES = [
    ("norm_one_row", W.EXIT_NORM, 1, 64, 50, 0, "bf16"),
    ("norm_ragged", W.EXIT_NORM, 5, 192, 1000, 0, "bf16"),
    ("norm_32_rows", W.EXIT_NORM, 32, 128, 777, 0, "bf16"),
    ("norm_70_rows", W.EXIT_NORM, 70, 64, 333, 0, "bf16"),
    ("norm_vocab_one", W.EXIT_NORM, 3, 64, 1, 0, "bf16"),
    ("embedding", W.EXIT_EMBEDDING, 9, 128, 500, 0, "bf16"),
    ("mlp", W.EXIT_MLP, 7, 192, 900, 320, "bf16"),
    ("norm_f32", W.EXIT_NORM, 6, 64, 333, 0, "f32"),
    ("mlp_f32", W.EXIT_MLP, 33, 128, 300, 192, "f32"),
    ("embedding_f32", W.EXIT_EMBEDDING, 2, 64, 129, 0, "f32"),
    ("layernorm_bias", W.EXIT_NORM, 9, 192, 1000, 0, "bf16"),
    ("layernorm_bias_f32", W.EXIT_NORM, 4, 64, 333, 0, "f32"),
    ("norm_max_hidden", W.EXIT_NORM, 3, 32768, 500, 0, "bf16"),
    ("mlp_max_hidden", W.EXIT_MLP, 5, 8192, 300, 256, "bf16"),
    # past 8 rows a weight of at least 12288 rows is read 64 rows a block:
    # the last block's second 32-row group lies past the vocabulary
    ("norm_wide_vocab", W.EXIT_NORM, 20, 128, 12300, 0, "bf16"),
    ("norm_wide_vocab_f32", W.EXIT_NORM, 12, 64, 12320, 0, "f32"),
    ("mlp_wide_inter", W.EXIT_MLP, 40, 128, 500, 12352, "bf16"),
    ("norm_max_vocab", W.EXIT_NORM, 3, 64, 1 << 20, 0, "bf16"),
]


@pytest.mark.parametrize("name,kind,n,h,v,inter,dtype", CASES, ids=[c[0] for c in CASES])
def test_small_decode_parity(name, kind, n, h, v, inter, dtype):
    say(f"case: decode {name} rows={n} h={h} V={v} I={inter} {dtype}")
    norm, bias = ("layer", True) if name.startswith("layernorm") else ("rms", False)
    w, b = make_case(kind, n, h, v, inter, dtype, seed=21, norm=norm, bias=bias)
    ex = O.exits_from_batch(b)[0]
    conf = D.exit_decide(ex, W.decode(b.hidden[0]), 0.5)["confidence"]
    thr = float(np.median(conf)) if n > 1 else 0.5
    check(b, thr, run_decide(b, thr))


def test_exact_tie_goes_to_lowest_id():
    # Rows 40 and 3000 of W_out identical and made dominant: both logits are
    # the same fp32 value on the device, so the lower id must win.
    w, b = make_case(W.EXIT_NORM, 4, 128, 5000, 0, "bf16", seed=22)
    z = O.exit_forward(O.exits_from_batch(b)[0], W.decode(b.hidden[0]))["z"]
    row = W.f32_to_bf16_bits((3.0 * z.mean(axis=0) / np.abs(z.mean(axis=0)).max()).astype(np.float32))
    b.exits[0].w_out[40] = row
    b.exits[0].w_out[3000] = row
    say("case: decode exact tie rows 40 and 3000")
    token, conf, flag = run_decide(b, 0.9)
    ref = check(b, 0.9, (token, conf, flag))
    tied = ref["logits"][:, 40] == ref["logits"].max(axis=1)
    assert tied.any()
    assert (token[tied] == 40).all()


def test_threshold_one_disables_exits():
    w, b = make_case(W.EXIT_NORM, 8, 64, 40, 0, "bf16", seed=23)
    # Row 7 of W_out along token 0's normalised state: token 0's top logit
    # leads by hundreds, so its probability is exactly 1.0 in fp32.
    z0 = O.exit_forward(O.exits_from_batch(b)[0], W.decode(b.hidden[0]))["z"][0]
    b.exits[0].w_out[7] = W.f32_to_bf16_bits((50.0 * z0 / np.abs(z0).max()).astype(np.float32))
    say("case: decode threshold 1")
    token, conf, flag = run_decide(b, 1.0)
    assert token[0] == 7 and conf[0] == 1.0
    assert not flag.any()
    token0, conf0, flag0 = run_decide(b, 0.0)
    assert flag0.all()


@pytest.mark.parametrize("rows", [1, 8, 32])
def test_full_size_decode(rows):
    # The 7B shape (h = 4096, V = 32000), Norm exit.
    say(f"case: decode full size rows={rows}")
    w, b = make_case(W.EXIT_NORM, rows, 4096, 32000, 0, "bf16", seed=24)
    ex = O.exits_from_batch(b)[0]
    conf = D.exit_decide(ex, W.decode(b.hidden[0]), 0.5)["confidence"]
    thr = float(np.median(conf))
    check(b, thr, run_decide(b, thr))


def test_full_size_mlp_decode():
    say("case: decode full-size MLP rows=4")
    w, b = make_case(W.EXIT_MLP, 4, 5120, 32000, 13824, "bf16", seed=25)
    check(b, 0.3, run_decide(b, 0.3))
