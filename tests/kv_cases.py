"""Case helpers shared by the cache-operation tests (CPU and GPU): no method
arithmetic, only slot bookkeeping from the block table and the generator's
packing."""
import numpy as np

from paper_2411_01142_amd import workloads as W

POISON = 0x7FC0  # bf16 quiet NaN


def last_token_slots(case):
    """(b, block id, slot) of token L-1 per request with L > 0, from the table."""
    out = []
    cap = case.max_blocks_per_seq * case.block_size
    for b, L in enumerate(case.seq_lens.tolist()):
        L = min(L, cap)
        if L <= 0:
            continue
        t = L - 1
        out.append((b, int(case.block_table[b, t // case.block_size]), t % case.block_size))
    return out


def drop_last_tokens(case):
    """Copy of ``case`` whose last tokens are poisoned, plus their (k, v) rows."""
    k_log, v_log = case.logical_kv()  # [NB][Hkv][bs][D]
    k_new = np.full((case.batch, case.num_kv_heads, case.head_dim), POISON, np.uint16)
    v_new = k_new.copy()
    for b, blk, slot in last_token_slots(case):
        k_new[b] = k_log[blk, :, slot, :]
        v_new[b] = v_log[blk, :, slot, :]
        k_log[blk, :, slot, :] = POISON
        v_log[blk, :, slot, :] = POISON
    dropped = W.Case(**{**case.__dict__, "k_cache": W.pack_k(k_log), "v_cache": W.pack_v(v_log)})
    return dropped, k_new, v_new


def used_blocks(case):
    """Sorted physical ids of the blocks the requests' tokens occupy."""
    cap = case.max_blocks_per_seq
    return sorted({int(x) for b, L in enumerate(case.seq_lens.tolist())
                   for x in case.block_table[b, :min((max(L, 0) + 15) // 16, cap)]})
