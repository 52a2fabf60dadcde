"""EFQ-Softmax attention forward for AMD Instinct MI355X (gfx950).

The compute path is the HIP library ``libefq_attn.so`` built from
``csrc/``; ``binding`` marshals arguments to its C ABI.
"""
