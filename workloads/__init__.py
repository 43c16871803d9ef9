"""Seeded synthetic workloads: layer shape tables and input generators.

Shared by the oracle tests, the GPU parity tests and the benchmark; holds no
quantized-operator arithmetic (see ``generate.py`` for the recipe)."""
from .shapes import (ConvLayer, DenseLayer, AddLayer, InvertedResidual, resnet50,
                     mobilenet_v2_blocks, mobilenet_v2_layers, inception_v3, bert_ffn,
                     SINGLE_CONV)
from .generate import (ConvCase, AddCase, single_conv_case, dense_case, conv_case,
                       add_case, sample_indices)
from .chain import (Chain, ChainConv, ChainAdd, ChainPool, resnet50_chain, mobilenet_v2_chain,
                    inception_v3_mixed5_chain)
