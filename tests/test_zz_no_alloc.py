"""seed_spec_forward_noalloc (the drafting-objective pass with its scratch in the library's fixed
array, for callers that cannot allocate) against seed_spec_forward (the same pass with a caller
buffer), through the C ABI: two calls in a row, the second with a smaller sequence, each equal
bit for bit to the buffered entry point's logits, per-row NLL and L_spec; a sequence that needs
more scratch than the array holds is refused."""
import numpy as np
import pytest

from gpu_common import decoder, say
from paper_2609_36590_amd import binding, synth

pytestmark = pytest.mark.gpu

TINY_BF16 = synth.C1_TINY.replace(name="tiny-4L-h256-bf16", dtype=synth.BF16)


@pytest.mark.parametrize("cfg", [synth.C1_TINY, TINY_BF16], ids=["f32", "bf16"])
def test_noalloc_equals_the_buffered_entry_point(cfg):
    import torch
    w = synth.make_weights(cfg, seed=0)
    dec = decoder(cfg, w, max_batch=1, max_ctx=128, max_draft=4)
    try:
        seqs = [synth.make_prompts(cfg.replace(prompt_len=n), seed=30 + n)[0] for n in (97, 41)]
        refs = [dec.spec_forward(x, 4) for x in seqs]
        # outputs allocated up front; the two no-alloc calls follow each other
        outs = [(torch.empty((len(x) - 1) * cfg.vocab, dtype=torch.float32, device="cuda"),
                 torch.empty(len(x) - 1, dtype=torch.float32, device="cuda")) for x in seqs]
        losses = []
        for x, (lg, nll) in zip(seqs, outs):
            say(f"[gpu] no-alloc spec forward {cfg.name} n={len(x)}")
            losses.append(binding.seed_spec_forward_noalloc(dec.ctx, x, 4, lg.data_ptr(), nll.data_ptr()))
        dec.stream.synchronize()
        for x, (lg, nll), loss, (lg_ref, nll_ref, loss_ref) in zip(seqs, outs, losses, refs):
            got = lg.cpu().numpy().reshape(len(x) - 1, cfg.vocab)
            assert np.all(np.isfinite(got))
            np.testing.assert_array_equal(got, lg_ref)
            np.testing.assert_array_equal(nll.cpu().numpy(), nll_ref)
            assert loss == loss_ref
    finally:
        dec.close()


def test_noalloc_refuses_sequences_beyond_its_scratch():
    # 4 KV heads x 64 dims x 4 bytes x 2 (keys, values) x 2 decoder layers = 4 KiB per position:
    # 16 MiB hold 4096 positions
    cfg = synth.C1_TINY
    w = synth.make_weights(cfg, seed=0)
    dec = decoder(cfg, w, max_batch=1, max_ctx=4200, max_draft=4)
    try:
        x = synth.make_prompts(cfg.replace(prompt_len=4100), seed=3)[0]
        import torch
        lg = torch.empty((len(x) - 1) * cfg.vocab, dtype=torch.float32, device="cuda")
        with pytest.raises(binding.SeedError) as e:
            binding.seed_spec_forward_noalloc(dec.ctx, x, 4, lg.data_ptr())
        assert e.value.status == -3 and "scratch" in str(e.value)
    finally:
        dec.close()
