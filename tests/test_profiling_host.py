"""Host logic of the profiling summaries: kernel names as rocprofv3 reports
them map to the short names used in profiles/ and by bench.py."""
from paper_2609_33916_amd import profiling


def test_short_names_of_backward_kernels():
    f = profiling.short_name
    assert f("void attn::dkdv16_kernel<128, true, 8, 64, false, false, 1>(attn::BwdArgs)") == "dkdv16_kernel"
    assert f("void attn::dkdv16_kernel<64, true, 4, 64, false, false, 2>(attn::BwdArgs)") == "dkdv16_kernel"
    assert f("void attn::dkdv16_kernel<128, false, 8, 64, true, false, 1>(attn::BwdArgs)") == "mat_dkdv16_kernel"
    assert f("void attn::dkdv16_kernel<64, true, 8, 64, false, true, 1>(attn::BwdArgs)") == "atomic_dq_dkdv16_kernel"
    assert f("void attn::dq_kernel<__bf16, 128, true, false>(attn::BwdArgs)") == "dq_kernel"
    assert f("void attn::dq_kernel<__bf16, 128, true, true>(attn::BwdArgs)") == "mat_dq_kernel"
    assert f("void attn::dkdv_kernel<float, 64, false, true>(attn::BwdArgs)") == "mat_dkdv_kernel"


def test_short_names_of_other_kernels():
    f = profiling.short_name
    assert f("void attn::fwd_kernel<__bf16, 128, true>(attn::FwdArgs)") == "fwd_kernel"
    assert f("void attn::fwd_pp_kernel<128, true>(attn::FwdArgs)") == "fwd_pp_kernel"
    assert f("void attn::mat_fwd_kernel<__bf16, 128, true>(attn::FwdArgs)") == "mat_fwd_kernel"
    assert f("void attn::decode_kernel<128>(attn::DecArgs)") == "decode_kernel"
    assert f("void attn::decode_combine_kernel<__bf16, 128>(float const*, void*, float*, int, int)") == \
        "decode_combine_kernel"
    assert f("void attn::bwd_prep_kernel<__bf16, 64>(attn::PrepArgs)") == "bwd_prep_kernel"
