"""bench.py's board power / clock summary: parsing of `amd-smi metric -p -c
--csv -w 1` output (CPU only, on a file in that format)."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402

HDR = ("timestamp,gpu,socket_power,gfx_voltage,gfx_0_clk,gfx_0_min_clk,gfx_0_max_clk,"
       "gfx_1_clk,gfx_1_min_clk,gfx_1_max_clk,mem_0_clk")


def sampler_on(tmp_path, text):
    p = tmp_path / "smi.csv"
    p.write_text(text)
    s = bench.PowerSampler.__new__(bench.PowerSampler)
    s.proc, s.path = None, str(p)
    return s


def test_window_median_and_xcd_mean(tmp_path):
    text = ("'CTRL' + 'C' to stop watching output:\n" + HDR + "\n"
            "99,0,240,N/A,95,500,2400,95,500,2400,1900\n\n" + HDR + "\n"
            "100,0,1300,N/A,1900,500,2400,1880,500,2400,1900\n"
            "101,0,1350,N/A,1890,500,2400,1870,500,2400,1900\n" + HDR + "\n"
            "102,0,1340,N/A,1896,500,2400,1884,500,2400,1900\n"
            "103,0,1340,N/A,18")  # a row cut off while written
    got = sampler_on(tmp_path, text).summary(100, 103)
    assert got["samples"] == 3
    assert got["socket_power_w"] == 1340.0
    # mean over the gfx_<i>_clk columns only (min/max clocks and other domains ignored)
    assert got["gfx_clk_mhz"] == 1890.0


def test_no_sample_in_window(tmp_path):
    text = HDR + "\n50,0,240,N/A,95,500,2400,95,500,2400,1900\n"
    assert sampler_on(tmp_path, text).summary(100, 110) is None


def test_sampler_declines_under_a_profiler(monkeypatch):
    """Under a profiler (whose preloaded tool library initialises the GPU in
    every process that inherits it) no child program is started."""
    import subprocess
    started = []
    monkeypatch.setattr(subprocess, "Popen", lambda *a, **k: started.append(a) or None)
    for env in ({"ROCPROF_OUTPUT_PATH": "/tmp/x"}, {"ROCPROFILER_LIBRARY_CTOR": "1"},
                {"ROCP_TOOL_LIBRARIES": "/opt/rocm/lib/x.so"}, {"HSA_TOOLS_LIB": "x.so"},
                {"LD_PRELOAD": "/opt/rocm/lib/librocprofiler-sdk-tool.so"}):
        assert bench.profiler_loaded(env)
        s = bench.PowerSampler(env=env)
        assert s.declined and s.proc is None and s.path is None
        assert s.summary(0, 1) is None
        s.close()
    assert started == []
    assert not bench.profiler_loaded({"PATH": "/usr/bin", "LD_PRELOAD": ""})


def test_sampler_runs_amd_smi_with_this_interpreter(monkeypatch):
    """Without a profiler the child is this interpreter running the amd-smi
    script (no exec of another program through its #! line)."""
    import shutil
    import subprocess
    calls = []

    class P:
        def __init__(self, argv, **kw):
            calls.append((argv, kw))

        def poll(self):
            return 0

    monkeypatch.setattr(shutil, "which", lambda name: "/opt/rocm/bin/amd-smi")
    monkeypatch.setattr(subprocess, "Popen", P)
    s = bench.PowerSampler(env={"PATH": "/usr/bin"})
    assert not s.declined and len(calls) == 1
    argv, kw = calls[0]
    assert argv[0] == sys.executable and argv[1] == "/opt/rocm/bin/amd-smi"
    assert not any(k.startswith("ROCP") for k in kw["env"])
    s.close()
