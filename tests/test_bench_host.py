"""Host logic of bench.py that needs no GPU: the power sampler and the energy arithmetic
(fed from a file that stands in for the hwmon sensor), and the refusal of N > 1."""
import subprocess
import sys
import time

import bench


class _FakeCuda:
    @staticmethod
    def synchronize():
        pass


class _FakeTorch:
    cuda = _FakeCuda


def test_power_sampler_reads_microwatts(tmp_path):
    f = tmp_path / "power1_input"
    f.write_text("250000000\n")
    with bench.PowerSampler(str(f), period=0.002) as ps:
        time.sleep(0.05)
    assert len(ps.samples) >= 5
    assert all(abs(w - 250.0) < 1e-9 for _, w in ps.samples)


def test_energy_is_mean_power_times_time_per_step(tmp_path):
    f = tmp_path / "power1_input"
    f.write_text("300000000\n")  # a constant 300 W

    def step():
        time.sleep(0.001)

    e = bench.measure_energy(_FakeTorch, step, 0.2, images=4, path=str(f))
    assert e["watts_mean"] == 300.0 and e["watts_idle"] == 300.0
    assert e["steps"] >= 10 and e["steps"] % 10 == 0
    # joules per step = W x wall seconds per step; per image divides by the batch
    assert abs(e["joules_per_step"] - 300.0 * e["seconds"] / e["steps"]) < 0.01 * e["joules_per_step"]
    assert abs(e["mj_per_image"] - 1e3 * e["joules_per_step"] / 4) < 0.01 * e["mj_per_image"]
    assert e["mj_per_image_above_idle"] == 0.0


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "4"], cwd=bench.ROOT, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_profile_tooling_names_compiled_kernels():
    """rocprof_report.kernel_symbol maps every persistent, streaming, whole-module and deep
    variant (and the split and int8 feature instances of the persistent ones) to a kernel
    the library contains, so that per-kernel statistics and traffic find their rows."""
    import os
    import re
    from paper_2404_19331_amd import fcm, rocprof_report
    lib = os.path.join(os.path.dirname(fcm.__file__), "libfcm.so")
    out = subprocess.run(["nm", "-C", lib], capture_output=True, text=True, check=True).stdout
    stubs = {m.group(1) for m in re.finditer(r"__device_stub__(k_\w+<[^>]*>)\(fcm::KArgs\)", out)}
    checked = 0
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not re.match(r"k_\w+[3567]<", name):
            continue
        forms = [dict()]
        if re.match(r"k_\w+3<", name):
            if not name.startswith("k_dw3<"):
                forms.append(dict(split=True))
            if "<i8," in name:
                forms += [dict(qx=1), dict(qx=2)] + ([dict(split=True, qx=1), dict(split=True, qx=2)]
                                                     if not name.startswith("k_dw3<") else [])
        for kw in forms:
            sym = rocprof_report.kernel_symbol(name, **kw)
            body = re.match(r"void fcm::(k_\w+<.*>)\(fcm::KArgs\)$", sym).group(1)
            assert body in stubs, (name, kw, sym)
            checked += 1
    assert checked > 50
