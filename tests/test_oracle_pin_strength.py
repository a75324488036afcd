"""The pins catch plausible mistakes: each test plants one mistake in a copy of
the oracle (on the CPU, never in the product) and requires that at least one
pin check fails on that copy."""
import importlib
import inspect
import types

import pytest

import oracle
oa = importlib.import_module("oracle.attention")
oe = importlib.import_module("oracle.edit_select")   # the package re-exports a function of that name
import oracle_pins as pins


def _mutant(module, old, new):
    src = inspect.getsource(module)
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    m = types.ModuleType(module.__name__ + "_mutant")
    exec(compile(src.replace(old, new), "<mutant>", "exec"), m.__dict__)
    return m


def _caught(checks, impl):
    for check in checks:
        try:
            check(impl)
        except Exception:          # AssertionError, or the mutant crashed on a shape
            return True
    return False


ATTN_MUTATIONS = {
    "block-causal sees one block too few": ("(i // block_size + 1) * block_size", "(i // block_size) * block_size"),
    "scale 1/D instead of 1/sqrt(D)": ("1.0 / math.sqrt(D)", "1.0 / D"),
    "softmax normalised over the whole matrix": ("E / E.sum(axis=1, keepdims=True)", "E / E.sum()"),
    "V page read token-major": ("v_pages[page, kv_head, :, slot]", "v_pages[page, kv_head, slot % v_pages.shape[2], :][:, :16]"),
    "interleaved GQA head mapping": ("range(g * G, (g + 1) * G)", "range(g, Hq, Hkv)"),
    "prefix hidden from the window": ("vis[i, :visible_count(", "vis[i, P:visible_count("),
    "window misses its last token": ("return prefix_len + window_len\n", "return prefix_len + window_len - 1\n"),
    "page index from slot": ("page_table_row)[t // PAGE_SIZE]", "page_table_row)[(t // PAGE_SIZE) // 2]"),
    "slot order reversed in page": ("slot = t % PAGE_SIZE", "slot = PAGE_SIZE - 1 - t % PAGE_SIZE"),
    "query rows not advanced per sequence": ("row0 += W", "row0 += 0"),
    "keys and queries swapped": ("S = scale * (Qb @ K.T)", "S = scale * (K[:W] @ Qb.T)[:, :1].repeat(n_all, 1)"),
}


@pytest.mark.parametrize("name", list(ATTN_MUTATIONS))
def test_attention_mutant_is_caught(name):
    old, new = ATTN_MUTATIONS[name]
    m = _mutant(oa, old, new)
    checks = pins.ATTENTION_CHECKS + [lambda impl: pins.check_brute_force(impl, oracle.brute_window_attention)]
    assert _caught(checks, m), f"no pin catches: {name}"


EDIT_MUTATIONS = {
    "argmax takes the last tie": ("a = int(np.argmax(row))", "a = int(len(row) - 1 - np.argmax(row[::-1]))"),
    "strict threshold": ("(c >= theta)", "(c > theta)"),
    "softmax without the max shift in the numerator": ("np.exp(row - row[a])", "np.exp(row)"),
    "edits even when argmax equals current": ("ch = (a != cur[r]) and (c >= theta)", "ch = (c >= theta)"),
    "overwrites regardless of the decision": ("new[r] = a if ch else cur[r]", "new[r] = a"),
    "confidence of the runner-up": ("c = 1.0 / np.sum(np.exp(row - row[a]))",
                                    "c = np.sort(np.exp(row - row[a]))[-2] / np.sum(np.exp(row - row[a]))"),
}


@pytest.mark.parametrize("name", list(EDIT_MUTATIONS))
def test_edit_mutant_is_caught(name):
    old, new = EDIT_MUTATIONS[name]
    m = _mutant(oe, old, new)
    assert _caught(pins.EDIT_CHECKS, m), f"no pin catches: {name}"


def test_unmutated_oracle_passes_all_pins():
    assert not _caught(pins.ATTENTION_CHECKS, oa)
    assert not _caught(pins.EDIT_CHECKS, oe)
