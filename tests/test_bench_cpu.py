"""bench.py's host logic without a GPU: the contract's refusal of more than
one GPU, and the mapping of rocprofv3's demangled kernel names onto the names
the library's own launch timer records."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_kernel_key_maps_profiler_names():
    k = bench.kernel_key
    assert k("void mpq::(anonymous namespace)::fit_hist_kernel<512, 9, true, true, false>"
             "(mpq::HistBatch)") == "fit_hist_kernel<512,9,lattice>"
    assert k("fit_hist_kernel<64, 2, true, false, false>(mpq::HistBatch)") == "fit_hist_kernel<64,2,linear>"
    assert k("fit_hist_kernel<256, 4, false, false, false>(x)") == "fit_hist_kernel<256,4,grid>"
    assert k("fit_hist_kernel<1024, 32, true, true, true>(x)") == "fit_hist_kernel<1024,32,lattice,rebuilt>"
    assert k("void mpq::(anonymous namespace)::gemm_err_kernel<true>(mpq::ErrGroup)") == "gemm_err_kernel"
    assert bench.stage_of("form_d_kernel") == "output_error"
    assert bench.stage_of("fit_hist_kernel<64,1,linear>") == "fit"
    assert bench.stage_of("zero_i32_kernel") is None
    assert k("void mpq::(anonymous namespace)::int_forward_kernel<0>(mpq::IntGroup)") == "int_forward_kernel<16>"
    assert k("int_forward_kernel<2>(mpq::IntGroup)") == "int_forward_kernel<1>"
    assert bench.stage_of("int_forward_kernel<16>") == "deploy"


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2 and "one GPU" in p.stderr
