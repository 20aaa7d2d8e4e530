"""Co-batched multi-LoRA linear layer (inference + LoRA fine-tuning tokens in one
batch) for AMD MI355X, after DeltaServe (arXiv 2607.28848).

The compute path is the HIP library libdsv.so behind include/dsv.h; its Python
binding is ``paper_2607_28848_amd.dsv`` (imported on demand: it raises when the
library is not built).  ``paper_2607_28848_amd.workloads`` draws the seeded
synthetic inputs.
"""
