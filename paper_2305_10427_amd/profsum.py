"""Condensed summaries of rocprofv3 CSV output for the decoder's kernels.

    python3 -m paper_2305_10427_amd.profsum kt  RUN_kernel_trace.csv
        per-kernel launches and durations per decoding iteration, counted from
        the first vocabulary launch on (the decode; the weight upload and the
        encoder come before it); then the same per-launch averages for each
        half of the decode's vocabulary launches (bench.py --decode-only
        decodes its sentences twice: graph replay, then the event-timed pass)
    python3 -m paper_2305_10427_amd.profsum pmc RUN_counter_collection.csv COUNTER
        per-kernel mean of COUNTER over the decode, and the three largest
        values of the runtime's copy kernel (the 256 MiB calibration copies
        bench.py --copy-calibration issues before anything else)

The last line of each summary is the same figures as one JSON object."""
import collections
import csv
import json
import sys


def _short(name):
    return name.split("(")[0].replace("void ", "")


def _decode_start(rows):
    return next(i for i, r in enumerate(rows) if "k_vocab" in r["Kernel_Name"])


def kernel_table(path):
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"]))
    dec = rows[_decode_start(rows):]
    iters = sum(1 for r in dec if "k_vocab" in r["Kernel_Name"])
    agg = collections.defaultdict(list)
    for r in dec:
        agg[_short(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    print(f"decoding iterations (vocabulary launches): {iters}")
    print("| kernel | launches / iteration | avg µs | µs / iteration |")
    print("|---|---|---|---|")
    total = 0.0
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        per = sum(v) / iters
        total += per
        if per >= 0.05:
            print(f"| `{k}` | {len(v) / iters:.2f} | {sum(v) / len(v):.2f} | {per:.1f} |")
    print(f"| sum of kernel durations | | | {total:.1f} |")
    vocab_at = [i for i, r in enumerate(dec) if "k_vocab" in r["Kernel_Name"]]
    cut = vocab_at[len(vocab_at) // 2] if len(vocab_at) >= 2 else len(dec)
    halves = {}
    for name, part in (("first half", dec[:cut]), ("second half", dec[cut:])):
        h = collections.defaultdict(list)
        for r in part:
            h[_short(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        prod = [x for k, v in h.items() if k.startswith("pdec::k_gemm") for x in v]
        halves[name] = {k: {"launches": len(v), "avg_us": round(sum(v) / len(v), 3)} for k, v in h.items()}
        halves[name]["all k_gemm"] = {"launches": len(prod), "avg_us": round(sum(prod) / max(len(prod), 1), 3)}
        print(f"{name}: k_gemm {len(prod)} launches, avg {sum(prod) / max(len(prod), 1):.2f} us; " +
              "; ".join(f"{k} avg {sum(v) / len(v):.2f} us" for k, v in h.items() if "k_vocab" in k or "k_attn" in k))
    print("JSON " + json.dumps({"iterations": iters, "kernels": {
        k: {"launches": len(v), "avg_us": round(sum(v) / len(v), 3)} for k, v in agg.items()}, "halves": halves}))


def counter_table(path, counter):
    rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    start = _decode_start(rows)
    copies = sorted(float(r["Counter_Value"]) for r in rows[:start] if "copyBuffer" in r["Kernel_Name"])[-3:]
    agg = collections.defaultdict(list)
    for r in rows[start:]:
        agg[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    print(f"{counter}: calibration copies (KiB per dispatch): {copies}")
    print(f"| kernel | dispatches | mean {counter} KiB |")
    print("|---|---|---|")
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{k}` | {len(v)} | {sum(v) / len(v):.1f} |")
    print("JSON " + json.dumps({"counter": counter, "copy_KiB": copies, "kernels": {
        k: {"dispatches": len(v), "mean_KiB": sum(v) / len(v)} for k, v in agg.items()}}))


if __name__ == "__main__":
    if len(sys.argv) >= 3 and sys.argv[1] == "kt":
        kernel_table(sys.argv[2])
    elif len(sys.argv) >= 4 and sys.argv[1] == "pmc":
        counter_table(sys.argv[2], sys.argv[3])
    else:
        sys.exit(__doc__)
