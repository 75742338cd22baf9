"""Plant plausible mistakes in a copy of the oracle and check the pins catch each.

Every mutation is a textual edit of the oracle's source, executed into a fresh
module on the CPU.  A mutation that no pin rejects would mean the pins leave
that part of the oracle unchecked.
"""

import inspect
import types

import pytest

import oracle.zeta_oracle as orc
import pins

MUTATIONS = {
    "bf16: wrong shift": ("<< np.uint32(16)).view(np.float32)", "<< np.uint32(15)).view(np.float32)"),
    "bf16: bits in the low half": ("astype(np.uint32) << np.uint32(16)).view(np.float32)",
                                   "astype(np.uint32) << np.uint32(0)).view(np.float32)"),
    "bf16: read as float16": ('    if dtype == "bf16":\n        return bf16_bits_to_f32(x)\n',
                              '    if dtype == "bf16":\n        return np.asarray(x, dtype=np.uint16).view(np.float16).astype(np.float32)\n'),
    "axis order reversed": ("d * s + (d - 1 - a)", "d * s + a"),
    "least significant bit first": ("d * s + (d - 1 - a)", "d * (bits - 1 - s) + (d - 1 - a)"),
    "grid of 2^b cells scale": ("top = np.float32((1 << bits) - 1)", "top = np.float32(1 << bits)"),
    "round instead of floor": ("c = np.clip(np.floor(w)", "c = np.clip(np.round(w)"),
    "range over queries only": ("both = np.concatenate([q, k], axis=1)", "both = q"),
    "no zero-range guard": ("w = np.where(den > np.float32(0), w, np.float32(0))", "w = np.nan_to_num(w)"),
    "unstable sort": ('perm = np.argsort(k_codes, axis=-1, kind="stable")',
                      'perm = np.argsort(k_codes.astype(np.int64) * 4096 - np.arange(k_codes.shape[-1]), axis=-1)'),
    "insertion on the right": ("p = bisect.bisect_left(pool, int(qc[i]) << 32)",
                               "p = bisect.bisect_right(pool, (int(qc[i]) << 32) | 0xFFFFFFFF)"),
    "searchsorted right": ('ps = np.searchsorted(sorted_codes, qc, side="left")',
                           'ps = np.searchsorted(sorted_codes, qc, side="right")'),
    "window leans right": ("s = min(max(p - k // 2, 0), pool_size - m)",
                           "s = min(max(p - (k + 1) // 2, 0), pool_size - m)"),
    "window truncated at end": ("s = min(max(p - k // 2, 0), pool_size - m)", "s = max(p - k // 2, 0)"),
    "diagonal excluded": ("    return i + 1\n", "    return i\n"),
    "chunk rule keeps own chunk": ("        return (i // chunk) * chunk\n", "        return min(n, (i // chunk + 1) * chunk)\n"),
    "chunk rule off by one": ("        return (i // chunk) * chunk\n", "        return (i // chunk) * chunk + 1\n"),
    "distance not squared": ("dist = np.sum(diff * diff, axis=-1)", "dist = np.sqrt(np.sum(diff * diff, axis=-1))"),
    "eps squared": ("score = np.where(valid, 1.0 / (dist + eps), 0.0)",
                    "score = np.where(valid, 1.0 / (dist + eps * eps), 0.0)"),
    "padding not masked": ("score = np.where(valid, 1.0 / (dist + eps), 0.0)", "score = 1.0 / (dist + eps)"),
    "not normalised": ("out[seg, r0:r0 + len(rr)] = num / zs[:, None]", "out[seg, r0:r0 + len(rr)] = num"),
    "bwd: o_i not subtracted": ('g = np.einsum("bd,bkd->bk", du, vj) - np.einsum("bd,bd->b", du, o)[:, None]',
                                 'g = np.einsum("bd,bkd->bk", du, vj)'),
    "bwd: delta not squared": ("w = np.where(valid, g / zs[:, None] / (delta * delta), 0.0)",
                               "w = np.where(valid, g / zs[:, None] / delta, 0.0)"),
    "bwd: not divided by Z": ("w = np.where(valid, g / zs[:, None] / (delta * delta), 0.0)",
                              "w = np.where(valid, g / (delta * delta), 0.0)"),
    "bwd: dq sign": ("dq[seg, rr] = -2.0 * np.einsum", "dq[seg, rr] = 2.0 * np.einsum"),
    "bwd: dq factor": ("dq[seg, rr] = -2.0 * np.einsum", "dq[seg, rr] = -1.0 * np.einsum"),
    "bwd: dk sign": ("(2.0 * w[:, :, None] * diff)", "(-2.0 * w[:, :, None] * diff)"),
    "bwd: dv unnormalised": ("(a[:, :, None] * du[:, None, :])", "(score[:, :, None] * du[:, None, :])"),
    "bwd: dv to query rows": ("np.add.at(dv[seg], jj.ravel()[sel]", "np.add.at(dv[seg], np.repeat(rr, jj.shape[1])[sel]"),
    "bwd: deps sign": ("deps -= float(w.sum())", "deps += float(w.sum())"),
    "bwd: padding not masked": ("score = np.where(valid, 1.0 / delta, 0.0)  # S_ij", "score = 1.0 / delta  # S_ij"),
    "query minus wrong row": ("diff = q[seg, rr][:, None, :] - k[seg][jj]  # [b, k, dk]",
                              "diff = q[seg, rr][:, None, :] - k[seg][rr][:, None, :]  # [b, k, dk]"),
    "bwd: query minus wrong row": ("diff = q[seg, rr][:, None, :] - k[seg][jj]  # q_i - k_j",
                                   "diff = q[seg, rr][:, None, :] - k[seg][rr][:, None, :]  # q_i - k_j"),
    "dot: no 1/sqrt(d)": ('return np.einsum("bd,bcd->bc", qr, keys) / np.sqrt(d)',
                          'return np.einsum("bd,bcd->bc", qr, keys)'),
    "neg_euclid: sign": ("return -dd / np.sqrt(d)", "return dd / np.sqrt(d)"),
    "norm_dot: keys not normalised": ('return np.einsum("bd,bcd->bc", unit(qr), unit(keys)) / np.sqrt(d)',
                                      'return np.einsum("bd,bcd->bc", unit(qr), keys) / np.sqrt(d)'),
    "inv_euclid: squared distance": ("return 1.0 / (np.sqrt(dd) + eps)", "return 1.0 / (dd + eps)"),
    "softmax: padding not masked": ("w = np.where(valid, np.exp(t - zmax[:, None]), 0.0)",
                                    "w = np.exp(t - zmax[:, None])"),
    "knn: ties not by position": ("order = np.lexsort((np.arange(end), d2))  # by distance, then position",
                                  "order = np.lexsort((-np.arange(end), d2))  # by distance, then position"),
    "knn: causal pool includes the future": ("            end = i + 1 if causal else N\n",
                                            "            end = min(N, i + 2) if causal else N\n"),
    "knn: unsquared distance": ("d2 = (d2 + (diff * diff).astype(np.float32)).astype(np.float32)",
                                "d2 = (d2 + np.abs(diff)).astype(np.float32)"),
    "overlap counts padding": ("set(int(x) for x in a2[r] if x >= 0) & set(int(x) for x in b2[r] if x >= 0)",
                               "set(int(x) for x in a2[r]) & set(int(x) for x in b2[r])"),
    "locality: wrong denominator": ("return float(index_overlap(win, nn).sum()) / float(np.count_nonzero(nn >= 0))",
                                    "return float(index_overlap(win, nn).sum()) / float(nn.size + 1)"),
    "history: sums instead of means": ("return np.cumsum(k, axis=1) / count, np.cumsum(v, axis=1) / count",
                                       "return np.cumsum(k, axis=1), np.cumsum(v, axis=1)"),
    "history: current row excluded": ("return np.cumsum(k, axis=1) / count, np.cumsum(v, axis=1) / count",
                                      "return (np.cumsum(k, axis=1) - k) / np.maximum(count - 1, 1), "
                                      "(np.cumsum(v, axis=1) - v) / np.maximum(count - 1, 1)"),
    "history: non-causal uses prefix": ("    mk = np.broadcast_to(k.mean(axis=1, keepdims=True), k.shape).copy()\n",
                                        "    mk = np.cumsum(k, axis=1) / np.arange(1, N + 1)[None, :, None]\n"),
    "history: mean not in normaliser": ("                z = z + sm\n", ""),
    "history: mean value unweighted": ("num = num + sm[:, None] * np.asarray(mean_v[seg, rr], dtype=np.float64)",
                                       "num = num + np.asarray(mean_v[seg, rr], dtype=np.float64)"),
    "history bwd: means not passed back": ("            dk += np.cumsum((dmk / count)[:, ::-1], axis=1)[:, ::-1]\n", ""),
    "history bwd: prefix instead of suffix": ("dv += np.cumsum((dmv / count)[:, ::-1], axis=1)[:, ::-1]",
                                              "dv += np.cumsum(dmv / count, axis=1)"),
    "history bwd: not divided by length": ("dv += np.cumsum((dmv / count)[:, ::-1], axis=1)[:, ::-1]",
                                           "dv += np.cumsum(dmv[:, ::-1], axis=1)[:, ::-1]"),
    "history bwd: mean missing from o": ("                o = o + a_m[:, None] * mean_v[seg, rr]\n", ""),
    "history bwd: dq term sign": ("dq[seg, rr] -= 2.0 * w_m[:, None] * dm", "dq[seg, rr] += 2.0 * w_m[:, None] * dm"),
    "history bwd: deps term missing": ("                deps -= float(w_m.sum())\n", ""),
    "history bwd: non-causal spread": ("dk += dmk.sum(axis=1, keepdims=True) / N", "dk += dmk / N"),
}


def _mutant(old, new):
    src = inspect.getsource(orc)
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    mod = types.ModuleType("zeta_oracle_mutant")
    exec(compile(src.replace(old, new), "zeta_oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_mutation(name):
    mod = _mutant(*MUTATIONS[name])
    caught = []
    for check in pins.ALL_PINS:
        try:
            check(mod)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            caught.append(check.__name__)
    assert caught, f"no pin rejects the planted mistake {name!r}"
