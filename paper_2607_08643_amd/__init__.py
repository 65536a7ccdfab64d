"""MI355X-native BSQ weight codec (BiSCo-LLM, arxiv 2607.08643): the encoder,
decoder assembly, fused decode-GEMV and fused decode-GEMM as hand-written HIP
for gfx950 behind the C ABI of include/bsq.h (libbsq.so), with a thin ctypes
binding whose functions carry the C names."""
from ._binding import (  # noqa: F401
    BSQ_BF16, BSQ_ERR_ALIGN, BSQ_ERR_ARG, BSQ_ERR_BUFFER_TOO_SMALL, BSQ_ERR_DEVICE, BSQ_ERR_DTYPE,
    BSQ_ERR_NONFINITE, BSQ_ERR_SHAPE, BSQ_ERR_UNSUPPORTED, BSQ_F32, BSQ_OK, DEC_IDENTITY, DEC_LINEAR,
    DEVERR_BAD_SET, DEVERR_NONFINITE, DEVERR_POISONED, DEVERR_TIMEOUT, ENC_IDENTITY, ENC_LINEAR, PROT_E4M3, PROT_E5M2,
    PROT_INT8,
    DEC_MLP, DEC_MLP_RES1, EXPORTS, LIB_PATH, OP_ENCODE, OP_GEMM, OP_GEMV, OP_SELECT, BsqError, Codec, Config, GemvPlan, Layer,
    bsq_codec_bytes, bsq_codec_prepare, bsq_config, bsq_config_check, bsq_coupled_select, bsq_debug_set_wait_limit,
    bsq_decode, bsq_decode_stage, bsq_decoder,
    bsq_encode, bsq_encode_with_set,
    bsq_gemm, bsq_gemv, bsq_gemv_noalloc, bsq_layer, bsq_layer_sizes, bsq_lora, bsq_sizes, bsq_version, bsq_workspace_bytes,
    TrainHyper, bsq_train_adam, bsq_train_grad, bsq_train_hparams, bsq_train_param_count, bsq_train_workspace_bytes,
    layer_empty, lib, status_str,
)
