"""bench.py's stage fractions cover every kernel of their stages: each
kernel the library can launch for the score and Gram contractions or for
the top-k and the compaction is in the stage's list, and the ones with
algorithmic units are in the work table."""
import importlib.util
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _library_kernel_names():
    text = open(os.path.join(ROOT, "paper_2606_07577_amd", "csrc", "api.hip")).read()
    table = text[text.index("kKernelNames[K_COUNT] = {"):]
    table = table[: table.index("};")]
    return re.findall(r'"([a-z_0-9]+)"', table)


def test_stage_lists_cover_the_library_kernels():
    b = _bench()
    names = _library_kernel_names()
    assert len(names) == len(set(names))
    select = [n for n in names if n.startswith(("psi_topk", "topk_")) or n in (
        "gather_compact", "gather_inplace", "stage_moved_back", "layer_inputs")]
    contractions = [n for n in names if n in ("lse_pass", "colsum_pass") or n.startswith("gram_")
                    and n not in ("gram_finish",)]
    assert set(select) <= set(b.TOPK_COMPACT_KERNELS), set(select) - set(b.TOPK_COMPACT_KERNELS)
    assert set(contractions) <= set(b.SCORE_GRAM_KERNELS), set(contractions) - set(b.SCORE_GRAM_KERNELS)
    assert set(b.TOPK_COMPACT_KERNELS) <= set(names) and set(b.SCORE_GRAM_KERNELS) <= set(names)


def test_work_table_units():
    b = _bench()
    score, gram, tin, tout, compact = b.layer_work(28, 2048, 4096, 4, 6144, 128, 2, 4608, 1536, 3500)
    work = b.work_table(score, gram, tin, tout, compact)
    for name in b.SCORE_GRAM_KERNELS:
        assert work[name][0] == "mfma" and work[name][1] > 0
    # every ranking path moves the same algorithmic bytes: a, s and modality in, idx out
    assert work["psi_topk"][1] == work["psi_topk_reg"][1] == work["topk_hist"][1] + work["topk_emit"][1] == tin + tout
    assert work["gather_compact"][1] == work["gather_inplace"][1] == compact == 2 * 2 * 4 * 3500 * 128 * 2
