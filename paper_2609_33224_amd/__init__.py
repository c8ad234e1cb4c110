"""MI355X (gfx950) window scorer for PackServe's KVC-first, SLO-aware request
packing.  The scoring path is the HIP library ``libpackserve.so`` behind the
C ABI of ``include/packserve.h``; :mod:`.binding` marshals its arguments."""
from .binding import (  # noqa: F401
    PS_F_FALLBACK_DCQ, PS_F_SELECTOR, PS_SEL_D, PS_SEL_DC, PS_SEL_DCQ, PS_SEL_DQ, PS_SEL_DQC,
    PS_SEL_HCQ, PS_SEL_LMETRIC, PS_SEL_RANDOM, PS_F_NO_KVC_FILTER, PS_F_NO_TPOT_FILTER, PS_F_TTFT_ADMIT, PS_R_FALLBACK, PS_R_INVALID,
    PS_R_REJECT, PS_R_TTFT_MISS, PS_REQ_DTYPE, PS_RESULT_DTYPE, PackServeError, PsModel, Scorer,
    load_library, make_model, pack_reqs, ps_build_id, ps_commit, ps_create, ps_destroy, ps_last_error,
    ps_load_instances, ps_probe_hits_dev, ps_read_state, ps_score_window, ps_score_window_dev,
    ps_schedule_window_dev, ps_replay_window_dev,
    ps_table_info, results_from_device, to_device_bytes, to_device_u64, ps_apply_events,
    ps_feedback_decode, ps_feedback_output, ps_read_model, PS_EV_PREFILL_DONE,
    PS_EV_DECODE_TOKENS, PS_EV_FINISHED, PS_LOUT_WINDOW,
)
