"""Test-side helpers: bf16 bit conversions and dense <-> paged placement.

These express the paged layout with numpy indexing (page, head, slot, dim
subscripts), independently of the flat index arithmetic in the oracle, so that
the oracle's address formula is checked against a second formulation.
"""
import numpy as np
import torch


def bf16_bits(x) -> np.ndarray:
    """fp32/fp64 values -> bf16 bit patterns (round to nearest even, by torch)."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bits_f64(bits) -> np.ndarray:
    """bf16 bit patterns -> float64 values (by torch's bf16 -> fp64 conversion)."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16)).view(np.int16)
    return torch.from_numpy(b.copy()).view(torch.bfloat16).to(torch.float64).numpy()


def randn_bits(rng: np.random.Generator, shape) -> np.ndarray:
    return bf16_bits(rng.standard_normal(shape))


def place(k_rows, v_rows, num_pages: int, Hkv: int, P: int, D: int, rng: np.random.Generator,
          extra_pages: int = 3, fill=None):
    """Put per-row dense K/V (lists of [Hkv][L_b][D] bit arrays) onto shuffled pages.

    Returns (k_pool, v_pool, block_table). K pages are [page][Hkv][P][D] and
    V pages [page][Hkv][D][P]. Pages no row owns, and the unused slots of a
    row's last page, are filled with `fill` bits (random if None).
    """
    B = len(k_rows)
    lens = [kr.shape[1] for kr in k_rows]
    pages = [(L + P - 1) // P for L in lens]
    total = sum(pages) + extra_pages
    assert total <= num_pages or num_pages == 0
    num_pages = max(num_pages, total)
    perm = rng.permutation(num_pages).astype(np.int32)
    stride = max(1, max(pages) if pages else 1)
    bt = np.zeros((B, stride), np.int32)
    if fill is None:
        k_pool = randn_bits(rng, (num_pages, Hkv, P, D))
        v_pool = randn_bits(rng, (num_pages, Hkv, D, P))
    else:
        k_pool = np.full((num_pages, Hkv, P, D), fill, np.uint16)
        v_pool = np.full((num_pages, Hkv, D, P), fill, np.uint16)
    off = 0
    for b in range(B):
        bt[b, :pages[b]] = perm[off:off + pages[b]]
        bt[b, pages[b]:] = perm[-1]          # unused entries: a page nobody owns
        off += pages[b]
        for j in range(lens[b]):
            pg, s = bt[b, j // P], j % P
            k_pool[pg, :, s, :] = k_rows[b][:, j, :]
            v_pool[pg, :, :, s] = v_rows[b][:, j, :]
    return k_pool, v_pool, bt


def dense_rows(k_pool, v_pool, bt, lens):
    """Inverse of place(): per-row [Hkv][L][D] bit arrays read through the block table."""
    P = k_pool.shape[2]
    ks, vs = [], []
    for b, L in enumerate(lens):
        j = np.arange(L)
        pg = bt[b, j // P]
        s = j % P
        ks.append(np.transpose(k_pool[pg, :, s, :], (1, 0, 2)))   # [Hkv][L][D]
        vs.append(np.transpose(v_pool[pg, :, :, s], (1, 0, 2)))   # [Hkv][L][D]
    return ks, vs
