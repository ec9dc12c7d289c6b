"""Validator of bench.py's JSON line against the measurement contract: the
fields the benchmark must report, their types, and the relations between
them (value and ms_per_step, the roofline fraction, the one-GPU rules)."""
import math

REQUIRED = {
    "metric": str, "value": (int, float), "unit": str, "n_gpus": int, "steps": int, "warmup": int,
    "ms_per_step": (int, float), "higher_is_better": bool, "scaling": str, "dtype": str, "data": str,
    "config": dict, "roofline": dict,
}
ROOFLINE = {"bound": str, "achieved": (int, float), "peak": (int, float), "unit": str, "frac": (int, float)}
CPU = {"value": (int, float), "unit": str, "cores": int, "kind": str, "sample": str}


def problems(line, want_cpu=True):
    """The contract violations of one parsed bench line (empty if none)."""
    bad = []
    for k, t in REQUIRED.items():
        if k not in line:
            bad.append("missing %s" % k)
        elif not isinstance(line[k], t) or (t is not bool and isinstance(line[k], bool)):
            bad.append("%s has type %s" % (k, type(line[k]).__name__))
    if bad:
        return bad
    if line["n_gpus"] != 1:
        bad.append("n_gpus %r (one GPU)" % line["n_gpus"])
    if "vs_baseline" not in line or line["vs_baseline"] is not None:
        bad.append("vs_baseline must be present and null (the paper gives no number for this metric)")
    if not line["value"] > 0 or not line["ms_per_step"] > 0:
        bad.append("value and ms_per_step must be positive")
    if "workload" not in line["config"]:
        bad.append("config.workload missing")
    if line["scaling"] not in ("weak", "strong"):
        bad.append("scaling %r" % line["scaling"])
    r = line["roofline"]
    for k, t in ROOFLINE.items():
        if k not in r or not isinstance(r[k], t):
            bad.append("roofline.%s missing or mistyped" % k)
    if "traffic" not in r:
        bad.append("roofline.traffic missing (null allowed)")
    if not bad:
        if r["bound"] not in ("hbm", "mfma", "alu"):
            bad.append("roofline.bound %r" % r["bound"])
        if not 0 < r["frac"] <= 1 or not math.isclose(r["frac"], r["achieved"] / r["peak"], rel_tol=2e-3, abs_tol=2e-4):
            bad.append("roofline.frac %r is not achieved / peak in (0, 1]" % r["frac"])
        if r["bound"] == "hbm" and (r["unit"] != "GB/s" or r["peak"] != 8000.0):
            bad.append("an HBM roofline is priced against 8000 GB/s")
        if r["traffic"] is not None and not r["traffic"] > 0:
            bad.append("roofline.traffic must be null or positive")
    if want_cpu:
        c = line.get("cpu_baseline")
        if not isinstance(c, dict):
            bad.append("cpu_baseline missing")
        else:
            for k, t in CPU.items():
                if k not in c or not isinstance(c[k], t):
                    bad.append("cpu_baseline.%s missing or mistyped" % k)
            if c.get("kind") != "oracle" or not c.get("cores", 0) >= 1:
                bad.append("cpu_baseline must be the oracle on >= 1 core")
    # images/s from the step time (the headline's unit)
    if line["unit"] == "images/s" and "images" in line["config"]:
        want = line["config"]["images"] / (line["ms_per_step"] * 1e-3)
        if not math.isclose(line["value"], want, rel_tol=2e-3):
            bad.append("value %r is not images / step time (%r)" % (line["value"], want))
    return bad
