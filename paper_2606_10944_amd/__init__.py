"""thin: MI355X-native thinned attention (kernel halving under kappa_att +
coreset attention), after "Express Language Modeling".

The compute path lives in the HIP library libthin.so (C ABI in include/thin.h);
this package only binds it.
"""
from ._lib import (THIN_BF16, THIN_EDTYPE, THIN_EHIP, THIN_EINVAL, THIN_EUNIFORMS,  # noqa: F401
                   THIN_EWORKSPACE, THIN_FP32, THIN_OK, ExpressCache, LaunchTimer, ThinError,
                   thin_attention, thin_compress, thin_express_plan, thin_express_prefill,
                   thin_express_prefill_plan, thin_plan,
                   thin_selftest_gram16, thin_status_str, workspace_status)
