"""The MQAR batches (Appendix C): N distinct keys and N distinct values per
example, the second half queries every key of the first half once, targets
are the paired values, and queries do not write."""
import torch

from paper_2609_36529_amd import mqar


def test_batch_structure():
    gen = torch.Generator().manual_seed(3)
    key_ids, val_ids, write, targets = mqar.make_batch(16, 37, gen)
    assert key_ids.shape == (16, 74) and targets.shape == (16, 37)
    for b in range(16):
        keys, vals = key_ids[b, :37], val_ids[b, :37]
        assert len(set(keys.tolist())) == 37 and len(set(vals.tolist())) == 37
        assert sorted(key_ids[b, 37:].tolist()) == sorted(keys.tolist())
        pair = dict(zip(keys.tolist(), vals.tolist()))
        assert [pair[k] for k in key_ids[b, 37:].tolist()] == targets[b].tolist()
        assert torch.all(val_ids[b, 37:] == -1)
        assert torch.all(write[b, :37] == 1) and torch.all(write[b, 37:] == 0)
    assert int(key_ids.max()) < mqar.N_KEYS and int(targets.max()) < mqar.N_VALS


def test_model_shapes_on_cpu_with_a_plain_mixer():
    """The model's plumbing (not the recurrence) with a stand-in mixer that
    returns zeros of the right shape: logits over the value vocabulary."""
    def zero_mixer(q, k, v, q2, k2, g, beta):
        return torch.zeros_like(v)
    model = mqar.MQARModel(4, zero_mixer)
    batch = mqar.make_batch(2, 8, torch.Generator().manual_seed(1))
    loss, acc = model.loss_acc(batch)
    assert loss.ndim == 0 and 0.0 <= acc.item() <= 1.0
