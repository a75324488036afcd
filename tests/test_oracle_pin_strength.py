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
import oracle_pins_next as pins_next
ou = importlib.import_module("oracle.update")
oen = importlib.import_module("oracle.entropy")
okv = importlib.import_module("oracle.kv_cache")


def _mutant(module, old, new):
    src = inspect.getsource(module)
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    m = types.ModuleType(module.__name__ + "_mutant")
    m.__package__ = "oracle"          # relative imports resolve against the real package
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
    "token-major V read token-minor": ("V = _f64(v_pages[page, kv_head, slot, :])",
                                       "V = _f64(v_pages[page, kv_head, :, slot % v_pages.shape[3]])"),
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


UPDATE_MUTATIONS = {
    "Gamma uses >= instead of >": ("if conf[r] > om:", "if conf[r] >= om:"),
    "force-unmask takes the last of equal confidences": ("if conf[r] > conf[best]:", "if conf[r] >= conf[best]:"),
    "force-unmask even when Gamma is not empty": ("if m_rows and not any(action[r] == UNMASK for r in m_rows):",
                                                  "if m_rows:"),
    "no force-unmask": ("            action[best] = FORCE_UNMASK", "            pass"),
    "edits masked rows too": ("        elif pred[r] != cur[r] and conf[r] >= oe:", "        if pred[r] != cur[r] and conf[r] >= oe:"),
    "edit ignores the threshold": ("elif pred[r] != cur[r] and conf[r] >= oe:", "elif pred[r] != cur[r]:"),
    "block flag from the first row only": ("1 if np.any(action[k * B:(k + 1) * B] != KEEP) else 0",
                                           "1 if action[k * B] != KEEP else 0"),
}


@pytest.mark.parametrize("name", list(UPDATE_MUTATIONS))
def test_update_mutant_is_caught(name):
    old, new = UPDATE_MUTATIONS[name]
    m = _mutant(ou, old, new)
    assert _caught(pins_next.UPDATE_CHECKS, m), f"no pin catches: {name}"


ENTROPY_MUTATIONS = {
    "entropy without the log-sum-exp": ("logp = fin - lse", "logp = fin - mx"),
    "entropy in bits": ("out[r] = -float(np.sum(np.exp(logp) * logp))", "out[r] = -float(np.sum(np.exp(logp) * logp)) / math.log(2.0)"),
    "tail size rounded down": ("k = int(math.ceil(float(np.float32(rho)) * B))", "k = max(1, int(float(np.float32(rho)) * B))"),
    "tail takes the smallest entropies": ("top = np.sort(e[i * B:(i + 1) * B])[::-1][:k]", "top = np.sort(e[i * B:(i + 1) * B])[:k]"),
    "selection ties go to the latest block": ("if best == j or S[b, i] > S[b, best]:", "if best == j or S[b, i] >= S[b, best]:"),
    "candidate window one block too wide": ("lo = max(0, j - int(k_max) + 1)", "lo = max(0, j - int(k_max))"),
    "current block is a candidate": ("for i in range(lo, j):", "for i in range(lo, j + 1):"),
}


@pytest.mark.parametrize("name", list(ENTROPY_MUTATIONS))
def test_entropy_mutant_is_caught(name):
    old, new = ENTROPY_MUTATIONS[name]
    m = _mutant(oen, old, new)
    assert _caught(pins_next.ENTROPY_CHECKS, m), f"no pin catches: {name}"


KV_MUTATIONS = {
    "V written token-major": ("V[page, :, :, slot] = vn[row]", "V[page, :, slot % V.shape[2], :] = vn[row][:, :16]"),
    "slot off by one": ("slot = pos % PAGE", "slot = (pos + 1) % PAGE"),
    "positions relative to the page start": ("pos = int(st[b]) + t", "pos = t"),
    "later-block mode refreshes nothing extra": ("elif seen and mode == REFRESH_CHANGED_AND_LATER:", "elif False:"),
    "page from the token index, not the position": ("page = int(pt[b, pos // PAGE])", "page = int(pt[b, t // PAGE])"),
    "start offset off by one": ("pos = int(st[b]) + t", "pos = int(st[b]) + t + 1"),
    "page stride of 8 tokens": ("page = int(pt[b, pos // PAGE])", "page = int(pt[b, min(pos // 8, pt.shape[1] - 1)])"),
    "K and V rows swapped": ("K[page, :, slot, :] = kn[row]", "K[page, :, slot, :] = vn[row]"),
    "block flags ignored": ("if fl is None or fl[b, t // int(block_size)]:", "if True:"),
    "block flag of the absolute position": ("fl[b, t // int(block_size)]",
                                            "fl[b, min((int(st[b]) + t) // int(block_size), fl.shape[1] - 1)]"),
    "rows counted only when written": ("                    V[page, :, :, slot] = vn[row]\n            row += 1",
                                       "                    V[page, :, :, slot] = vn[row]\n                row += 1"),
    "token-major V written token-minor": ("                    V[page, :, slot, :] = vn[row]",
                                          "                    V[page, :, :, slot] = vn[row][:, :16]"),
}


@pytest.mark.parametrize("name", list(KV_MUTATIONS))
def test_kv_mutant_is_caught(name):
    old, new = KV_MUTATIONS[name]
    m = _mutant(okv, old, new)
    assert _caught(pins_next.KV_CHECKS, m), f"no pin catches: {name}"


def test_unmutated_next_oracle_passes_all_pins():
    assert not _caught(pins_next.UPDATE_CHECKS, ou)
    assert not _caught(pins_next.ENTROPY_CHECKS, oen)
    assert not _caught(pins_next.KV_CHECKS, okv)
