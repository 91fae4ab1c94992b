"""Device memory for one decoder stack, held in torch tensors, driven through
the C ABI. torch provides allocations and streams only; all compute is in
libsidp."""

import torch

from . import (
    SIDP_STREAMED,
    make_config,
    sidp_create,
    sidp_decode_step,
    sidp_destroy,
    sidp_kv_attach,
    sidp_kv_region_bytes,
    sidp_layer_bytes,
    sidp_pool_bytes,
    sidp_slot_bytes,
    sidp_pool_init,
    sidp_pool_load_layer,
    sidp_set_pooling,
    sidp_sync,
)


def k_blocks_to_lib(k):
    """Key blocks from the natural layout [..., block, kv_head, token, d] to the
    library's [..., block, kv_head, d / 8, token, d % 8] (a view; copy_ it into
    the cache)."""
    *lead, bs, d = k.shape
    return k.reshape(*lead, bs, d // 8, 8).transpose(-3, -2)


def k_blocks_from_lib(kl):
    """Key blocks from the library's layout back to [..., block, kv_head, token, d]."""
    *lead, d8, bs, e = kl.shape
    return kl.transpose(-3, -2).reshape(*lead, bs, d8 * e)


class WaSDecoder:
    """A weight pool of num_layers packed layer blobs, a 2-slot weight cache,
    and num_regions paged KV regions of num_phys_blocks blocks each.

    cfg: mapping with num_layers, hidden, num_q_heads, num_kv_heads, head_dim,
    ffn_dim, qkv_bias, qk_norm, rms_eps, qk_norm_eps, rope_theta, block_size.
    """

    def __init__(self, cfg, max_batch, max_seq_len, num_phys_blocks, num_regions, device="cuda", slots=True):
        self.cfg = dict(cfg)
        self.device = torch.device(device)
        self.config = make_config(cfg, max_batch, max_seq_len)
        self.h = None
        self.h = sidp_create(self.config)
        self.layer_bytes = sidp_layer_bytes(self.config)
        self.pool = torch.empty(sidp_pool_bytes(self.config), dtype=torch.uint8, device=self.device)
        self.slots = torch.empty(sidp_slot_bytes(self.config), dtype=torch.uint8, device=self.device) if slots else None
        for t in (self.pool, self.slots):
            if t is not None and t.data_ptr() % 256:
                raise RuntimeError("device allocation is not 256-byte aligned")
        sidp_pool_init(self.h, self.pool, self.pool.numel(), self.slots,
                       0 if self.slots is None else self.slots.numel())
        self.num_phys_blocks = num_phys_blocks
        self.num_regions = num_regions
        region_elems = sidp_kv_region_bytes(self.config, num_phys_blocks) // 2
        self.k_cache = torch.empty(num_regions * region_elems, dtype=torch.bfloat16, device=self.device)
        self.v_cache = torch.empty(num_regions * region_elems, dtype=torch.bfloat16, device=self.device)
        sidp_kv_attach(self.h, self.k_cache, self.v_cache, num_phys_blocks, num_regions)

    # Cache views in the library's layouts.
    def k_view(self):
        """K blocks are stored [region][block][kv_head][d / 8][token][d % 8]."""
        c = self.cfg
        return self.k_cache.view(self.num_regions, self.num_phys_blocks, c["num_kv_heads"], c["head_dim"] // 8,
                                 c["block_size"], 8)

    def k_natural(self, region):
        """Region `region` of the K cache as [block][kv_head][token][d] (a copy)."""
        return k_blocks_from_lib(self.k_view()[region])

    def set_k_natural(self, region, k):
        """Writes key blocks given as [block][kv_head][token][d] into region `region`."""
        self.k_view()[region].copy_(k_blocks_to_lib(k))

    def v_view(self):
        """V blocks are stored transposed: [region][block][kv_head][d][token]."""
        c = self.cfg
        return self.v_cache.view(self.num_regions, self.num_phys_blocks, c["num_kv_heads"], c["head_dim"],
                                 c["block_size"])

    def load_layer(self, layer, weights, stream=None):
        sidp_pool_load_layer(self.h, layer, weights, stream)

    def set_pooling(self, mode, ranks=0, rank=0):
        """What a streamed layer stages (SIDP_POOL_LAYER / SIDP_POOL_FFN) and which
        layers this rank owns (l % ranks == rank); call between steps, after sync."""
        sidp_set_pooling(self.h, mode, ranks, rank)

    def step(self, hidden, positions, block_tables, flags=SIDP_STREAMED, compute=None, copy=None):
        compute = compute if compute is not None else torch.cuda.current_stream(self.device)
        sidp_decode_step(self.h, hidden, positions, block_tables, block_tables.shape[1], hidden.shape[0], flags,
                         compute, copy)

    def sync(self):
        sidp_sync(self.h)

    def close(self):
        if self.h is not None:
            sidp_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
