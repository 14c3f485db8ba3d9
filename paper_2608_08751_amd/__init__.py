"""MI355X-native IVF routing and construction hot path of InSituANN
(arXiv 2608.08751).

The computation lives in ``libivf.so`` (hand-written HIP for gfx950, C ABI in
``include/ivf.h``); this package is the thin Python binding used by the tests
and the benchmark:

* ``ivf_route``         coarse search, Eq. (1) with Eq. (6): top-nprobe lists per query;
* ``ivf_kmeans_step``   one Lloyd iteration: assignment + mean update;
* ``ivf_assign_build``  full assignment + cluster-major inverted lists;
* ``ivf_build_lists``   the inverted-list build alone.
"""
from ._binding import (  # noqa: F401
    IVF_EDEVICE,
    IVF_EINVAL,
    IVF_ENOMEM,
    IVF_EUNSUPPORTED,
    IVF_F32,
    IVF_OK,
    IVF_OP_ADC_SCAN,
    IVF_OP_ASSIGN_BUILD,
    IVF_OP_BUILD_LISTS,
    IVF_OP_KMEANS_STEP,
    IVF_OP_PQ_TRAIN_STEP,
    IVF_OP_ROUTE,
    IVF_OPT_ASSIGN_SLICE,
    IVF_OPT_BUILD_BLOCKS,
    IVF_OPT_FORCE_FALLBACK,
    IVF_OPT_FORCE_RESCREEN,
    IVF_OPT_FP32_SCREEN,
    IVF_OPT_I8_TWO_PLANE_ONLY,
    IVF_OPT_PROFILE,
    IVF_OPT_RESCREEN_CAP,
    IVF_OPT_S1_ID_ORDER,
    IVF_OPT_SAMPLE_RANK,
    IVF_OPT_SCREEN_WAVES,
    IVF_U8,
    LIB_PATH,
    SIGNATURES,
    Context,
    IvfError,
    ivf_assign_build,
    ivf_adc_scan,
    ivf_assign_cells,
    ivf_assign_graph,
    ivf_build_lists,
    ivf_kmeans_step,
    ivf_list_major,
    ivf_pq_encode,
    ivf_pq_train_step,
    ivf_route,
    ivf_route_noalloc,
    load_library,
)


def compile_library():
    """Compiles libivf.so for gfx950 (hipcc)."""
    from .build import build as _build

    return _build()
