"""CPU check of the single-launch decode layer's index arithmetic, on the
phase table and constants read from its source: every weight load of every
(workgroup, wave, step, lane) stays inside its tensor, each (row, K slice) is
computed exactly once, each output row is written once by the workgroup that
computed it, and the reduction and LDS indexes stay inside their arrays.
This guards the persistent kernel's loads before any launch."""
import os
import re

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_10183_amd", "csrc",
                   "q4_layer.hip")


def _constants():
    src = open(SRC).read()
    c = {}
    m = re.search(r"constexpr int kH = (\d+), kHq = (\d+), kHkv = (\d+), kI = (\d+);", src)
    c["kH"], c["kHq"], c["kHkv"], c["kI"] = map(int, m.groups())
    c["kWG"] = int(re.search(r"constexpr int kWG = (\d+);", src).group(1))
    c["kWaves"] = int(re.search(r"constexpr int kWaves = (\d+);", src).group(1))
    c["kSteps"] = int(re.search(r"constexpr int kSteps = (\d+);", src).group(1))
    body = re.search(r"constexpr PhaseShape kPh\[4\] = \{(.*?)\};", src, re.S).group(1)
    rows = re.findall(r"\{([^{}]*)\}", body)
    assert len(rows) == 4

    def val(e):
        for k, v in c.items():
            e = re.sub(rf"\b{k}\b", str(v), e)
        return int(eval(e, {"__builtins__": {}}))  # arithmetic of integer literals only

    keys = ("K", "N", "S", "P", "R", "C", "NT", "first")
    c["phases"] = [dict(zip(keys, [val(e) for e in r.split(",")])) for r in rows]
    m = re.search(r"constexpr int phase_of\(int step\) \{ return step < (\d+) \? 0 : \(step < (\d+) \? 1 : "
                  r"\(step < (\d+) \? 2 : 3\)\); \}", src)
    c["phase_bounds"] = tuple(map(int, m.groups()))
    assert re.search(r"uint32_t xs\[\(kI / kGroup\) \* 17\]", src), "LDS staging array declaration"
    c["xs_words"] = c["kI"] // 32 * 17
    return c


def test_fused_layer_index_arithmetic():
    c = _constants()
    kH, kHq, kHkv, kI, kWG, kWaves = c["kH"], c["kHq"], c["kHkv"], c["kI"], c["kWG"], c["kWaves"]
    b0, b1, b2 = c["phase_bounds"]
    phase_of = lambda st: 0 if st < b0 else 1 if st < b1 else 2 if st < b2 else 3
    rows_of = {"q": kHq, "k": kHkv, "v": kHkv, "o": kH, "gate": kI, "up": kI, "down": kH}
    K_of = {"q": kH, "k": kH, "v": kH, "o": kHq, "gate": kH, "up": kH, "down": kI}
    PH = c["phases"]
    assert PH[3]["first"] + PH[3]["C"] == c["kSteps"]
    for ph, P in enumerate(PH):
        G = P["K"] // 32
        assert P["S"] * P["P"] == kWaves and P["S"] * 64 >= G
        seen = {}
        for wg in range(kWG):
            for wave in range(kWaves):
                s, p = wave % P["S"], wave // P["S"]
                for i in range(P["C"]):
                    st = P["first"] + i
                    assert phase_of(st) == ph
                    local = p + P["P"] * i
                    row = wg * P["R"] + local
                    if not (local < P["R"] and row < P["N"]):
                        continue
                    if ph == 0:
                        t = "q" if row < kHq else ("k" if row < kHq + kHkv else "v")
                        lr = row - (0 if t == "q" else kHq if t == "k" else kHq + kHkv)
                        ts = [t]
                    else:
                        ts = ["o"] if ph == 1 else (["gate", "up"] if ph == 2 else ["down"])
                        lr = row
                    assert len(ts) == P["NT"]
                    for t in ts:
                        assert 0 <= lr < rows_of[t] and K_of[t] == P["K"]
                        # lane 63 is the largest group index of the wave
                        g = min(64 * s + 63, G - 1)
                        assert lr * (P["K"] // 2) + g * 16 + 16 <= rows_of[t] * P["K"] // 2
                        assert (lr * G + g) * 2 + 2 <= rows_of[t] * G * 2
                        assert rows_of[t] * P["K"] // 2 < 2 ** 31  # 32-bit buffer offsets
                    key = (row, s)
                    assert key not in seen, (ph, key)
                    seen[key] = (wg, wave, i)
        assert len(seen) == P["N"] * P["S"], (ph, len(seen))
        outs = set()
        for wg in range(kWG):
            for tid in range(P["P"] * P["C"]):
                pp, i = tid % P["P"], tid // P["P"]
                local = pp + P["P"] * i
                row = wg * P["R"] + local
                if local < P["R"] and row < P["N"]:
                    assert row not in outs
                    outs.add(row)
                    for s in range(P["S"]):
                        assert seen[(row, s)] == (wg, s + P["S"] * pp, i)
        assert outs == set(range(P["N"])), ph
        V = 4 if P["NT"] * P["C"] <= 4 else 8 if P["NT"] * P["C"] <= 8 else 16
        assert P["NT"] * P["C"] <= V and P["S"] * P["P"] * V <= kWaves * 16
        assert P["P"] * P["C"] <= kWaves * 64  # epilogue threads exist
    # grouped-query expansion of v (head_dim 128, 4 query heads per KV head) stays inside the attention output
    hd, ex = 128, kHq // kHkv
    assert max(((rv // hd) * ex + e) * hd + rv % hd for rv in range(kHkv) for e in range(ex)) < kHq
    # the LDS staging of a K-wide input: groups * 17 words for the widest input
    assert max(P["K"] for P in PH) // 32 * 17 <= c["xs_words"]
