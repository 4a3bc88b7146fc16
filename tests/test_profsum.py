"""Host logic of the profile summariser: bench frames are selected from a
kernel trace and counter runs by leg (cache reset) and frame (k_hist_key)."""
import csv
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

KERNELS = ["rn::k_hist_key<false>(rn::Dev)", "void rn::k_frame_plan<false>(rn::Dev)",
           "void rn::k_gru<false, true>(rn::Dev)", "void rn::k_score_finish<false, false>(rn::Dev)"]


def write_runs(tmp, legs):
    """A kernel trace and an MFMA counter run of `legs` legs; frame f of leg g
    has k_gru lasting 1000*(10*g + f + 1) ns and 7*(f+1) MFMA FLOPs."""
    trace, ctr = [], []
    i = 0

    def add(k, ns, flops=None):
        nonlocal i
        i += 1
        trace.append({"Dispatch_Id": i, "Kernel_Name": k, "Start_Timestamp": 100 * i,
                      "End_Timestamp": 100 * i + ns})
        ctr.append({"Dispatch_Id": i, "Kernel_Name": k, "Counter_Name": "MfmaFlopsF32",
                    "Counter_Value": flops or 0})
    add("void rn::k_pack_layer(rn::Dev)", 5)
    for g, nf in enumerate(legs):
        for _ in range(4):
            add("rn::k_fill_u32(unsigned int*, unsigned int, long long)", 3)
        for f in range(nf):
            add(KERNELS[0], 2000)
            add(KERNELS[1], 3000)
            add(KERNELS[2], 1000 * (10 * g + f + 1), 7 * (f + 1))
            add(KERNELS[3], 4000)
            if f == 1:
                add("rn::k_fold_stats(rn::Dev, long long*)", 9)
    for d, rows in (("t", trace), ("c", ctr)):
        os.makedirs(os.path.join(tmp, d), exist_ok=True)
        name = "run_kernel_trace.csv" if d == "t" else "run_counter_collection.csv"
        with open(os.path.join(tmp, d, name), "w", newline="") as fh:
            w = csv.DictWriter(fh, fieldnames=list(rows[0]))
            w.writeheader()
            w.writerows(rows)


def run(*args):
    return subprocess.run([sys.executable, "-m", "paper_1801_09866_amd.profsum", *args], cwd=ROOT,
                          capture_output=True, text=True)


def test_span_selects_the_timed_frames_of_the_first_leg(tmp_path):
    write_runs(str(tmp_path), [6, 6, 3])
    r = run("--span", "w", "--warmup", "2", "--steps", "3", "--trace", str(tmp_path / "t"),
            "--mfma", str(tmp_path / "c"))
    assert r.returncode == 0, r.stderr
    lines = r.stdout.splitlines()
    gru = next(l for l in lines if l.startswith("rn::k_gru"))
    # frames 2, 3, 4 of leg 0: 3, 4, 5 us
    assert gru.split()[1] == "3" and abs(float(gru.split()[2]) - 4.0) < 1e-9
    per = [l.split() for l in lines if l.split() and l.split()[0] in ("2", "3", "4")]
    assert [float(p[1]) for p in per] == [3.0, 4.0, 5.0]
    assert [float(p[2]) for p in per] == [21.0, 28.0, 35.0]


def test_span_of_a_later_leg_and_a_short_trace(tmp_path):
    write_runs(str(tmp_path), [6, 6, 3])
    r = run("--span", "w", "--warmup", "0", "--steps", "2", "--leg", "1", "--trace", str(tmp_path / "t"))
    assert r.returncode == 0, r.stderr
    gru = next(l for l in r.stdout.splitlines() if l.startswith("rn::k_gru"))
    assert abs(float(gru.split()[2]) - 11.5) < 1e-9
    r = run("--span", "w", "--warmup", "2", "--steps", "2", "--leg", "2", "--trace", str(tmp_path / "t"))
    assert r.returncode != 0 and "fewer than 4" in r.stderr


def test_span_over_several_legs_averages_them(tmp_path):
    write_runs(str(tmp_path), [6, 6, 6])
    r = run("--span", "w", "--warmup", "1", "--steps", "2", "--leg", "1,2", "--trace", str(tmp_path / "t"),
            "--mfma", str(tmp_path / "c"))
    assert r.returncode == 0, r.stderr
    lines = r.stdout.splitlines()
    gru = next(l for l in lines if l.startswith("rn::k_gru"))
    # frames 1, 2 of legs 1 and 2: 12, 13, 22, 23 us
    assert gru.split()[1] == "4" and abs(float(gru.split()[2]) - 17.5) < 1e-9
    per = [l.split() for l in lines if l.split() and l.split()[0] in ("1", "2")]
    assert [float(p[1]) for p in per] == [17.0, 18.0]
