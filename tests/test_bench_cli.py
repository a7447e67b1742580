"""bench.py's command line on the CPU: the one-GPU contract and its flags."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout == ""


def test_help_lists_the_contract_flags():
    r = _bench("--help")
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--settle-ms", "--per-workload",
                 "--lmhead-positions", "--no-cpu-baseline", "--plan-sweep"):
        assert flag in r.stdout, flag


def test_traffic_from_counter_runs(tmp_path):
    """The HBM traffic of the fused step: each counter's KiB per dispatch,
    scaled by what it reads for the 1 GiB elementwise add."""
    head = "Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n"
    add = "void at::native::vectorized_elementwise_kernel<16, at::native::CUDAFunctorOnSelf_add<unsigned char> >(int)"
    fused = "void fdllm::k_fused<fdllm::VecBf16x8, 4, 8, 2, false>(...)"
    (tmp_path / "f.csv").write_text(
        head + f'1,"{add}",FETCH_SIZE,524288\n2,"{fused}",FETCH_SIZE,4000000\n'
        f'3,"{fused}",FETCH_SIZE,4000002\n4,"elementwise_kernel<CUDAFunctorOnSelf_add<float> >",FETCH_SIZE,7\n')
    (tmp_path / "w.csv").write_text(
        head + f'1,"{add}",WRITE_SIZE,1048576\n2,"{fused}",WRITE_SIZE,800\n')
    out = tmp_path / "t.json"
    r = _bench("--traffic-from", str(tmp_path / "f.csv"), str(tmp_path / "w.csv"),
               "--traffic-out", str(out))
    assert r.returncode == 0, r.stderr
    import json
    t = json.loads(out.read_text())
    assert t["fetch_scale"] == 2.0 and t["write_scale"] == 1.0
    assert t["hbm_bytes_per_launch"] == (4000001 * 2.0 + 800) * 1024
    assert t["dispatches"] == {"fetch": {"copy": 1, "fused": 2}, "write": {"copy": 1, "fused": 1}}


def test_source_digest_ignores_comments_and_layout():
    sys.path.insert(0, ROOT)
    import bench
    a = 'int f(int x) { // twice\n  return 2 * x; /* done */ }\nconst char* s = "// kept";\n'
    b = 'int f(int x) {\n\n    return 2 * x;   }\nconst char* s = "// kept";  // the literal stays\n'
    c = 'int f(int x) { return 3 * x; }\nconst char* s = "// kept";\n'
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)
    assert '"// kept"' in bench._code_only(a)
