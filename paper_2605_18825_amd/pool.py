"""Device-resident block pool: torch tensors in the layout of include/sae.h.

Marshalling only.  The block type tau is computed on the device by
sae_block_type; child counts are the number of valid children per parent.
"""
import numpy as np
import torch

from . import api


class DevicePool:
    """Pool arrays of n_inst instances x N blocks on `device`."""

    def __init__(self, n_inst, N, device="cuda"):
        self.n_inst, self.N = n_inst, N
        T = n_inst * N
        d = device
        self.last_access = torch.zeros(T, dtype=torch.int32, device=d)
        self.meta = torch.zeros(T, dtype=torch.int16, device=d)
        self.off = torch.zeros(T, dtype=torch.int32, device=d)
        self.hash = torch.zeros(T, dtype=torch.int64, device=d)
        self.parent = torch.full((T,), -1, dtype=torch.int32, device=d)
        self.child_count = torch.zeros(T, dtype=torch.int32, device=d)
        self.ref_count = torch.zeros(T, dtype=torch.int32, device=d)
        self.access_count = torch.zeros(T, dtype=torch.int32, device=d)

    def bind(self, ctx):
        api.sae_bind_pool(ctx, self.last_access, self.meta, self.off, self.hash, self.parent,
                          self.child_count, self.ref_count, self.access_count)

    def fill_instance(self, inst, p, device="cuda"):
        """Fill instance `inst` from a synthetic pool dict (numpy arrays)."""
        N = self.N
        sl = slice(inst * N, (inst + 1) * N)
        dev = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a)).to(device=device, dtype=dt)
        counts = dev(p["counts"], torch.uint8).reshape(N, 5).contiguous()
        tau = torch.empty(N, dtype=torch.uint8, device=device)
        api.sae_block_type(counts, tau)
        parent = dev(p["parent"], torch.int32)
        valid = dev(p["valid"], torch.bool)
        kids = torch.zeros(N, dtype=torch.int32, device=device)
        has = (parent >= 0) & valid
        kids.index_add_(0, parent[has].long(), torch.ones(int(has.sum()), dtype=torch.int32, device=device))
        ref = dev(p["ref_count"], torch.int32)
        meta = api.pack_meta(dev(p["queue"], torch.int32), tau.to(torch.int32), dev(p["ntok"], torch.int32),
                             valid=valid, leaf=(kids == 0), ref=(ref > 0))
        self.meta[sl] = api.meta_to_u16(meta)
        self.last_access[sl] = dev(p["last_access"], torch.int32)
        self.off[sl] = api.off_to_u32(api.pack_off(dev(p["ob"], torch.int64), dev(p["omax"], torch.int64)))
        self.hash[sl] = dev(np.asarray(p["hash"], np.uint64).view(np.int64), torch.int64)
        self.parent[sl] = parent
        self.child_count[sl] = kids
        self.ref_count[sl] = ref
        self.access_count[sl] = dev(p.get("access_count", np.zeros(N, np.int32)), torch.int32)
        return tau


class SelectBuffers:
    """Output buffers of sae_score_select for n_inst instances, Q queues."""

    def __init__(self, n_inst, Q, max_k, device="cuda"):
        self.victims = torch.full((n_inst, Q, max_k), -1, dtype=torch.int32, device=device)
        self.scores = torch.zeros((n_inst, Q, max_k), dtype=torch.float32, device=device)
        self.count = torch.zeros((n_inst, Q), dtype=torch.int32, device=device)
        self.decision = torch.full((n_inst, max_k), -1, dtype=torch.int32, device=device)
        self.decision_count = torch.zeros(n_inst, dtype=torch.int32, device=device)

    def run(self, ctx, now, k, flags=0, k_per_inst=None, stream=None):
        api.sae_score_select(ctx, now, k, flags, self.victims, self.count, self.decision, self.decision_count,
                             scores=self.scores, k_per_inst=k_per_inst, stream=stream)

    def run_after_match(self, ctx, hashes, lens, pm_now, pm_flags, match_len, now, k, flags=0, matched_ids=None,
                        inst=None, k_per_inst=None, stream=None):
        """A prefix match, then this selection, in one sae_match_select call."""
        api.sae_match_select(ctx, hashes, lens, pm_now, pm_flags, match_len, now, k, flags, self.victims, self.count,
                             self.decision, self.decision_count, matched_ids=matched_ids, inst=inst,
                             scores=self.scores, k_per_inst=k_per_inst, stream=stream)
