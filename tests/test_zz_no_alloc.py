"""The allocation-free attention backward matches the workspace entry point.

enc_attn_bwd_noalloc runs the same kernels as enc_attn_bwd with the D vector
in the library's static per-GPU scratch instead of a caller workspace.  Two
calls in a row, the second on a smaller input (the scratch keeps the first
call's contents), must each equal enc_attn_bwd on the same inputs bit for
bit; a size past the scratch is refused before anything is launched.
"""

import pytest
import torch

from helpers import announce
from paper_2408_03505_amd import binding as B
from paper_2408_03505_amd.synthetic import random_bf16

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _inputs(batch, seq, heads, d, seed):
    M, A = batch * seq, heads * d
    qkv = random_bf16((M, 3 * A), seed).cuda()
    do = random_bf16((M, A), seed + 1).cuda()
    o, lse = B.enc_attn_fwd(batch, seq, heads, d, qkv)
    return qkv, o, lse, do


def test_noalloc_attention_backward_matches_workspace_entry_point():
    shapes = [(8, 256, 48, 128), (3, 33, 2, 80)]  # the second call is smaller
    for i, (b, s, h, d) in enumerate(shapes):
        announce(f"attn bwd noalloc vs workspace, call {i}: batch={b} seq={s} heads={h} head_dim={d}")
        qkv, o, lse, do = _inputs(b, s, h, d, seed=40 + i)
        ref = B.enc_attn_bwd(b, s, h, d, qkv, o, lse, do)
        got = torch.full_like(ref, float("nan"))
        B.enc_attn_bwd_noalloc(b, s, h, d, qkv, o, lse, do, got)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), (i, b, s, h, d)


def test_noalloc_attention_backward_refuses_past_the_scratch():
    b, s, h, d = 256, 257, 16, 64  # batch*heads*seq = 1052672 > 2^20
    announce("attn bwd noalloc size refusal (no launch)")
    M, A = b * s, h * d
    qkv = torch.empty((M, 3 * A), dtype=torch.bfloat16, device="cuda")
    o = torch.empty((M, A), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((b, h, s), dtype=torch.float32, device="cuda")
    dqkv = torch.empty_like(qkv)
    with pytest.raises(B.EncError) as e:
        B.enc_attn_bwd_noalloc(b, s, h, d, qkv, o, lse, o, dqkv)
    assert e.value.status == B.ENC_ERR_UNSUPPORTED and "static scratch" in str(e.value)
