"""Runs GPU parity cases through the bounds-checked build (libattuner_checked.so),
then corrupts block-table entries on purpose and checks that the checked
kernels report them and skip them.

Started by tests/test_gpu_checked.py as its own process with
ATTUNER_LIB_VARIANT=checked, so every binding call goes to the checked
library.  Prints one line per case ("[case] ..." before, "[ok] ..." after) and
exits non-zero at the first failure.

The planted entries stay inside the buffers the unchecked kernels would touch
(a page id one past the pool of layer 0 of a two-layer pool addresses layer
1's first page; destination rows past the end of a head's cache plane run into
the next head's plane), so the case is memory-safe even if a check were
missing: the test then fails on its assertions, not on a fault.
"""

import os
import sys
import traceback

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import ctypes as C  # noqa: E402

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2609_36722_amd import _lib  # noqa: E402

VIOL_GATHER_PAGE, VIOL_GATHER_ROWS, VIOL_COPY_ENTRY = 1 << 0, 1 << 1, 1 << 4

# (module, test function, arguments): the parity cases rerun on the checked build
CASES = [
    ("test_gpu_parity", "test_gather_c1_bit_exact", ()),
    ("test_gpu_parity", "test_gather_ragged_multilayer_multirequest_bit_exact", ()),
    ("test_gpu_parity", "test_gather_layers_split_from_table_bit_exact", ()),
    ("test_gpu_parity", "test_pool_reuse_after_release_bit_exact", ()),
    ("test_gpu_parity", "test_attention_random_batches", (101,)),
    ("test_gpu_parity", "test_suffix_layer_varlen_batch", ()),
    ("test_gpu_parity", "test_encode_store_assemble_equals_full_prefill", ()),
    ("test_gpu_gather_attn", "test_gather_attn_three_layers_bit_exact", ()),
    ("test_gpu_gather_attn", "test_gather_attn_short_suffixes", ()),
    ("test_gpu_gather_attn", "test_gather_attn_host_pages_fall_back", ()),
    ("test_gpu_decode", "test_decode_ragged_batch", ()),
    ("test_gpu_decode", "test_decode_random_batches", (201,)),
    ("test_gpu_spans", "test_interleaved_random_prompts", (301,)),
    ("test_gpu_host_pool", "test_staged_assembly_bit_exact", ()),
]


def say(tag, msg):
    print(f"[{tag}] {msg}", flush=True)


def violations(reset=True) -> int:
    bits = C.c_uint32(0)
    st = _lib.lib().attuner_bounds_violations(0, 1 if reset else 0, C.byref(bits))
    assert st == 0, f"attuner_bounds_violations: status {st}: {_lib.lib().attuner_last_error()}"
    return bits.value


def planted_entries():
    """Corrupted block-table entries given to attuner_gather_layers and to the
    attention launch's page copy: each is flagged and leaves the cache alone."""
    from synthdata.workloads import ModelShape, Request, custom_workload
    from tests._gpu import GpuWorkload

    wl = custom_workload("checked-plant", 71, ModelShape(hidden=2560), [1500, 700],
                         [Request((0, 1), 512)], n_layers=2, rank=8, scale=1.0, gamma="uniform")
    g = GpuWorkload(wl, layers=(0, 1))
    try:
        pool_pages = g.ctx.pool_info()[0]
        good = g.cache_view().copy()
        table = g.block_table.view(-1, 4).cpu().numpy().copy()
        sentinel = torch.full_like(g.req_kv, 0.5)
        assert violations() == 0

        # a page id one past the pool, then rows past the end of the plane
        for what, bit, edit in [("page id past the pool", VIOL_GATHER_PAGE, lambda t: t.__setitem__((0, 0), pool_pages)),
                                ("rows past the cache plane", VIOL_GATHER_ROWS,
                                 lambda t: t.__setitem__((1, 2), g.rows - 8))]:
            say("case", f"planted gather entry: {what}")
            bad = table.copy()
            edit(bad)
            # the runtime takes only the table of the last assembly: plant in it
            g.block_table.copy_(torch.from_numpy(bad.reshape(-1)))
            kv = sentinel.clone()
            g.ctx.gather_layers(g.block_table, g.n_entries, 0, 1, kv, g.rows)
            g.block_table.copy_(torch.from_numpy(table.reshape(-1)))
            got = violations()
            assert got == bit, f"{what}: violation bits {got:#x}, expected {bit:#x}"
            view = kv.view(torch.int16).cpu().numpy().reshape(good.shape)
            ref = good.view(np.int16)
            half = np.int16(0x3F00)  # bf16 0.5
            e = 0 if bit == VIOL_GATHER_PAGE else 1
            page, n_valid, dst = table[e, 0], table[e, 1], table[e, 2]
            # the skipped entry's rows keep the sentinel in every plane of layer 0
            assert (view[0, :, :, dst:dst + n_valid] == half).all(), f"{what}: the skipped entry was written"
            # every other entry of layer 0 was gathered as usual
            for j in range(g.n_entries):
                if j == e:
                    continue
                d, n = table[j, 2], table[j, 1]
                assert (view[0, :, :, d:d + n] == ref[0, :, :, d:d + n]).all(), f"{what}: entry {j} differs"
            say("ok", f"planted gather entry: {what} (bits {got:#x}, entry {e} of page {page} skipped)")

        # the page copy carried by the attention launch (layer 1's attention
        # copies layer 0's pages) with a page id past the pool
        say("case", "planted copy entry in attuner_suffix_attn_gather")
        from tests.test_gpu_gather_attn import _call, _qkv

        bad = table.copy()
        bad[0, 0] = pool_pages
        g.block_table.copy_(torch.from_numpy(bad.reshape(-1)))
        kv = g.req_kv.clone()
        kv.view(2, -1)[0].fill_(0.5)  # layer 0's planes: only the copy may write them
        ins = _qkv(g, 1)
        _call(g, 1, ins, kv, gather_layer=0, bt=g.block_table)
        got = violations()
        g.block_table.copy_(torch.from_numpy(table.reshape(-1)))
        # 512 suffix rows over 2200 cached keys: enough key tiles that the copy
        # rides in the attention launch (a short range would get a gather
        # launch of its own, reported as VIOL_GATHER_PAGE)
        assert got == VIOL_COPY_ENTRY, f"carried copy: violation bits {got:#x}, expected {VIOL_COPY_ENTRY:#x}"
        view = kv.view(torch.int16).cpu().numpy().reshape(good.shape)
        ref = good.view(np.int16)
        d0, n0 = table[0, 2], table[0, 1]
        assert (view[0, :, :, d0:d0 + n0] == np.int16(0x3F00)).all(), "carried copy: the skipped entry was written"
        for j in range(1, g.n_entries):  # every other entry copied as usual
            d, n = table[j, 2], table[j, 1]
            assert (view[0, :, :, d:d + n] == ref[0, :, :, d:d + n]).all(), f"carried copy: entry {j} differs"
        say("ok", f"planted copy entry (bits {got:#x})")
    finally:
        g.close()


def main() -> int:
    assert _lib.VARIANT == "checked", "run with ATTUNER_LIB_VARIANT=checked"
    flag = C.c_int32(-1)
    assert _lib.lib().attuner_bounds_checked(C.byref(flag)) == 0 and flag.value == 1, "not the checked build"
    assert torch.cuda.is_available(), "needs a GPU"
    say("info", f"library {_lib.LIB_PATH}")
    violations()  # start from a clear word
    import importlib

    for mod, fn, args in CASES:
        name = f"{mod}.{fn}{args if args else ''}"
        say("case", name)
        try:
            getattr(importlib.import_module(f"tests.{mod}"), fn)(*args)
        except Exception:
            traceback.print_exc()
            say("fail", name)
            return 1
        got = violations()
        if got != 0:
            say("fail", f"{name}: violation bits {got:#x} on valid input")
            return 1
        say("ok", name)
    try:
        planted_entries()
    except Exception:
        traceback.print_exc()
        say("fail", "planted entries")
        return 1
    say("done", f"{len(CASES)} parity cases and the planted entries")
    return 0


if __name__ == "__main__":
    sys.exit(main())
