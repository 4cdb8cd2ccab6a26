"""MI355X-native Allegro channel-wise tensor product (arxiv 2504.16068, §II.D).

The compute lives in liballegro_tp.so (hand-written HIP for gfx950 behind the
C ABI of include/allegro_tp.h and include/allegro_layer.h); this package is its
build script and a thin ctypes binding with the same entry-point names.  Importing the binding raises
if the library has not been built: there is no CPU fallback.
"""

from .binding import (  # noqa: F401
    ALLEGRO_DETERMINISTIC,
    ALLEGRO_E_HIP,
    ALLEGRO_E_INVALID,
    ALLEGRO_E_NOMEM,
    ALLEGRO_E_TIMEOUT,
    ALLEGRO_E_UNSUPPORTED,
    ALLEGRO_FULL_PARITY,
    ALLEGRO_OK,
    ALLEGRO_VALIDATE,
    AllegroError,
    Plan,
    allegro_env_embed,
    allegro_last_error,
    allegro_layer_backward,
    allegro_layer_buffers,
    allegro_layer_forward,
    allegro_sh_backward,
    allegro_sh_forward,
    allegro_tp_backward,
    allegro_tp_backward_train,
    allegro_tp_backward_train_noalloc,
    allegro_tp_backward_workspace,
    allegro_tp_forward,
    allegro_tp_plan_create,
    allegro_tp_plan_destroy,
    layer_weight_shapes,
)
